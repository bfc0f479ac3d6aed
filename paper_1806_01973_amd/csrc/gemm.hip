// Dense layers of CONVOLVE on gfx950 matrix cores (Algorithm 1):
//   line 1 over every pin once (Sec. 3.4):  P = ReLU(H Q^T + q)
//   lines 2-3:  h' = normalize(ReLU([h_self | n] W^T + w))
// as one templated MFMA GEMM  C = epi(A B^T + bias), A [M x K] assembled from
// two row sources (self rows through an optional row map, then the pooled
// rows), B [N x K] with a row stride (the PyTorch Linear layout of Q and W,
// or a column block of W).
//
// Work split: a block of WAVES_M x WAVES_N waves owns a BM x BN output tile;
// each wave owns (BM/WAVES_M) x (BN/WAVES_N), i.e. TM x TN blocks of 32 x 32.
//
// K pipeline: K runs in chunks of 64 bytes per row (32 bf16 / 16 fp32
// columns). Chunks travel global -> LDS by DMA (global_load_lds_dwordx4, no
// register staging) into a ring of STAGES LDS stages, STAGES - 1 chunks ahead
// of the MFMAs; one barrier per chunk. A stage packs rows in groups of 16; one
// DMA instruction of a wave fills one group (1 KB, row r of the group at
// 64 r): lanes 4r .. 4r+3 carry the four 16-byte vectors of row r, so a quad
// of lanes reads one contiguous 64-byte piece of a row. Inside a row, vector v
// sits in slot v ^ f(r), f(r) = ((r >> 1) ^ (r >> 3)) & 3, which spreads the
// 16 (resp. 8) rows of one LDS fragment read over distinct banks. Missing rows
// and the K tail read a static zero row, so loads never branch.
//
// fp32 storage: v_mfma_f32_32x32x2_f32; step st of a chunk pairs half-wave h
// with chunk column 8h + st (two 16-byte reads per fragment). bf16 storage:
// v_mfma_f32_32x32x16_bf16 (gfx950); k-step ks takes vector 2ks + h. fp32
// accumulation in both cases. The weight fragment is the MFMA's first
// operand, so the accumulators hold C^T blocks: a lane owns one output row
// and runs of 4 adjacent output columns, stored as one 8-byte (bf16) or
// 16-byte (fp32) vector.
//
// Epilogue: + bias, + an optional addend matrix (the pooled neighbour term
// when W is split, see run_layer), ReLU (optional without L2), store in the
// storage dtype; with L2 the block spans
// all N columns, and a row's sum of squares is added over the lane's own
// columns, its partner half-wave and then the waves of the row band in a fixed
// order through LDS; every row is scaled by 1/||z|| (zero rows stay zero).
//
// Tile order is XCD-aware: hardware hands block b to XCD b % 8; blocks are
// renumbered so that each XCD gets a contiguous run of tiles, keeping the
// column tiles of one row block on one XCD's L2.
#include <type_traits>

#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// A row of zeros as long as the widest A row (d_in + m <= 16384 fp32): rows
// that do not exist and the K tail read from here. Never written.
constexpr int kMaxGemmK = 16384;
__device__ __attribute__((aligned(16))) float g_zero_row[kMaxGemmK];

constexpr int kChunkRowBytes = 64;   // bytes of one row per K chunk
constexpr int kGroupBytes = 1024;    // 16 rows x 64 bytes: one DMA instruction

// Slot of 16-byte vector v of row r (r mod 16) inside the row's 64 bytes.
__device__ __forceinline__ int vec_slot(int r, int v) { return v ^ (((r >> 1) ^ (r >> 3)) & 3); }

template <bool BF16, int BM_, int BN_, int WAVES_M_, int WAVES_N_, bool L2_, int STAGES_>
struct Cfg {
  static constexpr bool kBf16 = BF16;
  static constexpr bool kTwoSources = L2_;  // the W layer reads [h_self | n]
  static constexpr bool L2 = L2_;
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
  static constexpr int NWAVES = WAVES_M * WAVES_N;
  static constexpr int THREADS = 64 * NWAVES;
  static constexpr int STAGES = STAGES_;
  static constexpr int ESZ = BF16 ? 2 : 4;       // bytes per element
  static constexpr int VEC = 16 / ESZ;            // elements per 16-byte vector
  static constexpr int BK = kChunkRowBytes / ESZ; // K columns per chunk
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int A_GROUPS = BM / 16;
  static constexpr int GROUPS = (BM + BN) / 16;
  static constexpr int DPW = GROUPS / NWAVES;     // DMA instructions per wave per chunk
  static constexpr int PENDING = (STAGES - 2) * DPW;
  static constexpr int STAGE_BYTES = GROUPS * kGroupBytes;
  static constexpr int RED_BYTES = L2 ? WAVES_N * BM * 4 : 0;
  static constexpr int BIAS_BYTES = BN * 4;
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES + RED_BYTES + BIAS_BYTES;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile is a multiple of 32x32");
  static_assert(GROUPS % NWAVES == 0, "every wave issues the same DMA count");
  static_assert(STAGES >= 2 && PENDING <= 63, "vmcnt range");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget of one workgroup");
};

__device__ __forceinline__ int xcd_tile(int b, int nt) {
  const int per = nt / 8, rem = nt % 8;
  const int xcd = b % 8, slot = b / 8;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// One 16-byte-per-lane DMA from global memory into LDS: lane l's vector lands
// at byte lds_base + 16 l (lds_base wave-uniform, via M0).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds_base), "v"(g)
               : "memory");
}

// Waits until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// Workgroup barrier after this wave's LDS operations have completed.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory");
}

template <typename C>
__global__ __launch_bounds__(C::THREADS) void gemm_kernel(GemmLaunch a) {
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, VEC = C::VEC;
  constexpr int TM = C::TM, TN = C::TN, THREADS = C::THREADS, ESZ = C::ESZ;
  constexpr int DPW = C::DPW, STAGES = C::STAGES;
  // LDS: the stage ring, then the cross-wave row-norm partials and the
  // block's bias slice.
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS_BYTES];
  float* red = reinterpret_cast<float*>(smem + STAGES * C::STAGE_BYTES);
  float* bias_s = reinterpret_cast<float*>(smem + STAGES * C::STAGE_BYTES + C::RED_BYTES);
  const uint32_t smem_base =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int64_t m0 = (int64_t)(tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;
  const int K = a.K0 + a.K1;
  // Bias slice of the block (zero past N).
  for (int c = tid; c < BN; c += THREADS)
    bias_s[c] = (a.bias && n0 + c < a.N) ? a.bias[n0 + c] : 0.0f;
  const int64_t ldb = a.ldb ? a.ldb : K;

  // ---- DMA slots (fixed across the K loop) --------------------------------
  // Slot d of this wave fills group wave*DPW + d of every stage: A groups
  // first, then B groups. Lane l serves row 16 * group + (l >> 2) and LDS
  // slot l & 3 of it, i.e. column vector vec_slot(l >> 2, l & 3). Source-1
  // pointers are biased by -K0 columns so both sources take the column kk;
  // rows that do not exist point at the zero row.
  const unsigned char* const zrow = reinterpret_cast<const unsigned char*>(g_zero_row);
  const int64_t k0b = (int64_t)a.K0 * ESZ;
  const unsigned char* p0[DPW];
  const unsigned char* p1[C::kTwoSources ? DPW : 1];
#pragma unroll
  for (int d = 0; d < DPW; ++d) {
    const int grp = wave * DPW + d;
    const int rr = lane >> 2;
    if (grp < C::A_GROUPS) {
      const int64_t gr = m0 + grp * 16 + rr;
      const bool in_m = gr < a.M;
      const int64_t src = !in_m ? -1 : (a.rowmap ? (int64_t)a.rowmap[gr] : gr);
      p0[d] = (src >= 0 && src < a.rows_a0)
                  ? static_cast<const unsigned char*>(a.A0) + src * a.lda0 * ESZ
                  : zrow;
      if constexpr (C::kTwoSources) {
        const unsigned char* q = (in_m && a.A1)
                                     ? static_cast<const unsigned char*>(a.A1) + gr * a.lda1 * ESZ
                                     : zrow;
        p1[d] = reinterpret_cast<const unsigned char*>(reinterpret_cast<uintptr_t>(q) - k0b);
      }
    } else {
      const int r = n0 + (grp - C::A_GROUPS) * 16 + rr;
      p0[d] = r < a.N ? static_cast<const unsigned char*>(a.B) + (int64_t)r * ldb * ESZ : zrow;
      if constexpr (C::kTwoSources) p1[d] = p0[d];
    }
  }
  const int kvec = vec_slot(lane >> 2, lane & 3) * VEC;
  const int nchunks = (K + BK - 1) / BK;
  // Tiles start their K sweep at different chunks (rotation by the tile's
  // index in the whole product):
  // rows of A and B sit at power-of-two strides, and blocks that all read the
  // same K columns at once would pile onto a few L2 channels.
#ifndef PINSAGE_GEMM_KSHIFT
#define PINSAGE_GEMM_KSHIFT 0
#endif
  const int64_t abs_tile = tile + (a.row_base / BM) * tiles_n;
  const int kshift = PINSAGE_GEMM_KSHIFT == 0 ? (int)(abs_tile % nchunks)
                     : PINSAGE_GEMM_KSHIFT == 1 ? 0
                     : (int)((abs_tile / tiles_n) % nchunks);
  // Issues the DMAs of the chunk-th chunk of this tile's sweep into its
  // stage. Sweep positions past the end read the zero row, which keeps the
  // in-flight count uniform for wait_vmcnt.
  auto issue = [&](int chunk) __attribute__((always_inline)) {
    int kc = chunk + kshift;
    kc = chunk >= nchunks ? nchunks : (kc >= nchunks ? kc - nchunks : kc);
    const int kk = kc * BK + kvec;
    const bool kin = kk < K;
    const int64_t off = (int64_t)kk * ESZ;
    const uint32_t dst = smem_base + (uint32_t)((chunk % STAGES) * C::STAGE_BYTES) +
                         (uint32_t)(wave * DPW * kGroupBytes);
#pragma unroll
    for (int d = 0; d < DPW; ++d) {
      const unsigned char* p;
      if constexpr (C::kTwoSources) p = (kk < a.K0 ? p0[d] : p1[d]) + off;
      else p = p0[d] + off;
      dma16(kin ? p : zrow, __builtin_amdgcn_readfirstlane(dst + d * kGroupBytes));
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int row_in_blk = lane & 31;
  const int half = lane >> 5;
  const int a_base_row = wm * C::WM;
  const int b_base_row = wn * C::WN;
  // Byte offset of a lane's fragment row (block-relative row r of A, resp.
  // B) in a stage. Fragment rows start at multiples of 32, so the row's place
  // in its group (lane & 15) and hence its vector slots depend on the lane.
  auto frag_off = [&](int r) __attribute__((always_inline)) {
    return (r >> 4) * kGroupBytes + (r & 15) * kChunkRowBytes;
  };
  const int fa_off = frag_off(a_base_row + row_in_blk);
  const int fb_off = C::A_GROUPS * kGroupBytes + frag_off(b_base_row + row_in_blk);
  // Byte offset of the vector a lane reads in half-step hs.
  auto vec_off = [&](int hs) __attribute__((always_inline)) {
    const int v = C::kBf16 ? 2 * hs + half : 2 * half + hs;
    return vec_slot(lane & 15, v) * 16;
  };
  const int voff0 = vec_off(0), voff1 = vec_off(1);

  // A chunk is multiplied in two half-steps hs = 0, 1. bf16: half-step hs is
  // the MFMA k-step hs, half-wave h reads column vector 2hs + h. fp32: MFMA
  // steps 4hs .. 4hs+3, half-wave h reads vector 2h + hs (column 8h + st).
  constexpr int FW = 4;  // 32-bit words per fragment per half-step
  typedef uint32_t frag_t __attribute__((ext_vector_type(FW)));
  struct Frags {
    frag_t a[TM], b[TN];
  };
  auto read_frags = [&](const unsigned char* stage, int hs, Frags& f)
      __attribute__((always_inline)) {
    const int v = hs ? voff1 : voff0;
#pragma unroll
    for (int i = 0; i < TM; ++i)
      f.a[i] = *reinterpret_cast<const frag_t*>(stage + fa_off + i * 2 * kGroupBytes + v);
#pragma unroll
    for (int j = 0; j < TN; ++j)
      f.b[j] = *reinterpret_cast<const frag_t*>(stage + fb_off + j * 2 * kGroupBytes + v);
  };
  auto mfma_half = [&](const Frags& f) __attribute__((always_inline)) {
    if constexpr (C::kBf16) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, f.b[j]), __builtin_bit_cast(bf16x8, f.a[i]), acc[i][j],
              0, 0, 0);
    } else {
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                __uint_as_float(f.b[j][st]), __uint_as_float(f.a[i][st]), acc[i][j], 0, 0, 0);
    }
  };
  auto stage_of = [&](int chunk) __attribute__((always_inline)) {
    return smem + (chunk % STAGES) * C::STAGE_BYTES;
  };

  // Ring protocol: chunks 0..STAGES-2 are in flight before the loop. Before
  // the fragments of chunk c+1 are read, each wave waits for its DMAs of that
  // chunk (STAGES - 2 younger chunks may stay in flight) and for its own LDS
  // reads of chunk c, then a barrier makes all DMAs visible and frees chunk
  // c's stage, which receives chunk c + STAGES. The half-step MFMAs issued
  // just before the barrier keep the matrix pipe busy across it.
#pragma unroll
  for (int c = 0; c < STAGES - 1; ++c) issue(c);
  wait_vmcnt<C::PENDING>();
  lds_barrier();
  issue(STAGES - 1);
  Frags f0, f1;
  read_frags(stage_of(0), 0, f0);
  // The last chunk is peeled off so the loop body has no branch: every
  // half-step's fragment reads then have a known count of younger reads.
  // Scheduling barriers pin the order: fragment reads go out right before a
  // half-step's 16 MFMAs that hide their latency.
  for (int c = 0; c + 1 < nchunks; ++c) {
    read_frags(stage_of(c), 1, f1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_half(f0);
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<C::PENDING>();
    lds_barrier();
    read_frags(stage_of(c + 1), 0, f0);
    __builtin_amdgcn_sched_barrier(0);
    issue(c + STAGES);
    __builtin_amdgcn_sched_barrier(0);
    mfma_half(f1);
    __builtin_amdgcn_sched_barrier(0);
  }
  read_frags(stage_of(nchunks - 1), 1, f1);
  mfma_half(f0);
  mfma_half(f1);
  wait_vmcnt<0>();  // drain the zero-row DMAs issued past the end
  __syncthreads();  // bias slice (and, below, row partials) visible

  // ---- epilogue -----------------------------------------------------------
  // Lane l: output row m0 + a_base_row + 32i + l%32; for group g of tile j,
  // output columns c0(j, g) + 0..3 with c0 = b_base_row + 32j + 8g + 4(l/32)
  // inside the block. N is a multiple of 16, so a group is all in or all out;
  // columns past N have zero weights and zero bias, so they stay zero.
  // Row bands are finished one at a time to keep few accumulators live.
  auto c0 = [&](int j, int g) __attribute__((always_inline)) { return b_base_row + j * 32 + 8 * g + 4 * half; };
  // bf16 tiles that fit in the (now free) stage ring are staged there, rows
  // padded by 16 bytes, and leave as whole rows (16 bytes per lane) rather
  // than as 8-byte pieces of 32 rows per store instruction. (Loading the
  // addend tile the same way, in front of the epilogue, measured slower: its
  // latency is then exposed.)
  constexpr int TROW = BN * 2 + 16;
  constexpr bool kStaged = C::kBf16 && BM * TROW <= STAGES * C::STAGE_BYTES;
  constexpr int PER_ROW = BN / 8;  // 16-byte pieces per tile row
  // + bias (+ addend), then ReLU unless disabled; the L2 epilogue always
  // follows a ReLU.
  const bool relu = a.relu || C::L2;
  auto bias_relu = [&](int i) __attribute__((always_inline)) {
    const int rt = a_base_row + i * 32 + row_in_blk;
    const int64_t r = m0 + rt;
    const bool add = a.addend != nullptr && r < a.M;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 bv = *reinterpret_cast<const float4*>(bias_s + c0(j, g));
        float x[4] = {acc[i][j][4 * g + 0] + bv.x, acc[i][j][4 * g + 1] + bv.y,
                      acc[i][j][4 * g + 2] + bv.z, acc[i][j][4 * g + 3] + bv.w};
        const int c = n0 + c0(j, g);
        if (add && c < a.N) {
          const int64_t o = r * a.N + c;
          if constexpr (C::kBf16) {
            const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.addend) + o);
            x[0] += __uint_as_float(v.x << 16);
            x[1] += __uint_as_float(v.x & 0xFFFF0000u);
            x[2] += __uint_as_float(v.y << 16);
            x[3] += __uint_as_float(v.y & 0xFFFF0000u);
          } else {
            const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(a.addend) + o);
            x[0] += v.x;
            x[1] += v.y;
            x[2] += v.z;
            x[3] += v.w;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][4 * g + e] = relu ? fmaxf(x[e], 0.0f) : x[e];
      }
  };
  auto store_band = [&](int i, float scale) __attribute__((always_inline)) {
    const int rt = a_base_row + i * 32 + row_in_blk;  // row in the tile
    const int64_t r = m0 + rt;
    if (!kStaged && r >= a.M) return;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = n0 + c0(j, g);
        const float v0 = acc[i][j][4 * g] * scale, v1 = acc[i][j][4 * g + 1] * scale;
        const float v2 = acc[i][j][4 * g + 2] * scale, v3 = acc[i][j][4 * g + 3] * scale;
        if constexpr (kStaged) {
          *reinterpret_cast<uint2*>(smem + rt * TROW + c0(j, g) * 2) =
              make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
        } else {
          if (c >= a.N) continue;
          const int64_t o = r * a.N + c;
          if constexpr (C::kBf16) {
            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.C) + o) =
                make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
          } else {
            *reinterpret_cast<float4*>(static_cast<float*>(a.C) + o) =
                make_float4(v0, v1, v2, v3);
          }
        }
      }
  };
  // Staged tile -> global, BN / 8 lanes per row.
  auto flush_tile = [&]() __attribute__((always_inline)) {
    if constexpr (kStaged) {
      __syncthreads();
#pragma unroll 4
      for (int e = tid; e < BM * PER_ROW; e += THREADS) {
        const int rt = e / PER_ROW, ck = e % PER_ROW;
        const int64_t r = m0 + rt;
        const int c = n0 + 8 * ck;
        if (r < a.M && c < a.N)
          *reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.C) + r * a.N + c) =
              *reinterpret_cast<const uint4*>(smem + rt * TROW + 16 * ck);
      }
    }
  };

  // bf16 L2 tiles too large to stage whole (512 columns): one row band at a
  // time through the free stage ring, so the addend arrives and the output
  // leaves as whole 16-byte row pieces (consecutive lanes, consecutive
  // pieces of a row) instead of 8-byte pieces of 32 rows per instruction.
  // Band i is row band i of every wave: tile rows WM wm' + 32 i + (0..31) for
  // each wm'; band row b <-> tile row WM (b / 32) + 32 i + b % 32.
  constexpr bool kBandLds = C::kBf16 && C::L2 && !kStaged;
  constexpr int BROWS = 32 * C::WAVES_M;
  static_assert(!kBandLds || BROWS * TROW <= STAGES * C::STAGE_BYTES, "a band fits the ring");
  auto band_row = [&](int i, int b) __attribute__((always_inline)) {
    return (b >> 5) * C::WM + 32 * i + (b & 31);
  };

  if constexpr (!C::L2) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      bias_relu(i);
      store_band(i, 1.0f);
    }
    flush_tile();
  } else if constexpr (kBandLds) {
    const int b_lane = wm * 32 + row_in_blk;  // this lane's row within a band
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      // The band's addend rows into LDS (rows past M read as zeros).
      if (a.addend) {
#pragma unroll 4
        for (int e = tid; e < BROWS * PER_ROW; e += THREADS) {
          const int b = e / PER_ROW, ck = e % PER_ROW;
          const int64_t r = m0 + band_row(i, b);
          const int c = n0 + 8 * ck;
          uint4 v = make_uint4(0u, 0u, 0u, 0u);
          if (r < a.M && c < a.N)
            v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.addend) + r * a.N + c);
          *reinterpret_cast<uint4*>(smem + b * TROW + 16 * ck) = v;
        }
      }
      __syncthreads();
      // + bias + addend, ReLU, and the row's partial sum of squares.
      float s = 0.0f;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 bv = *reinterpret_cast<const float4*>(bias_s + c0(j, g));
          float x[4] = {acc[i][j][4 * g + 0] + bv.x, acc[i][j][4 * g + 1] + bv.y,
                        acc[i][j][4 * g + 2] + bv.z, acc[i][j][4 * g + 3] + bv.w};
          if (a.addend) {
            const uint2 v = *reinterpret_cast<const uint2*>(smem + b_lane * TROW + c0(j, g) * 2);
            x[0] += __uint_as_float(v.x << 16);
            x[1] += __uint_as_float(v.x & 0xFFFF0000u);
            x[2] += __uint_as_float(v.y << 16);
            x[3] += __uint_as_float(v.y & 0xFFFF0000u);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[i][j][4 * g + e] = fmaxf(x[e], 0.0f);
        }
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) s = fmaf(acc[i][j][e], acc[i][j][e], s);
      s += __shfl_xor(s, 32);
      if (half == 0) red[wn * BM + a_base_row + i * 32 + row_in_blk] = s;
      __syncthreads();  // partial sums visible; every addend read of the band done
      {
        const int r = a_base_row + i * 32 + row_in_blk;
        float ss = 0.0f;
#pragma unroll
        for (int w = 0; w < C::WAVES_N; ++w) ss += red[w * BM + r];
        const float scale = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const float v0 = acc[i][j][4 * g] * scale, v1 = acc[i][j][4 * g + 1] * scale;
            const float v2 = acc[i][j][4 * g + 2] * scale, v3 = acc[i][j][4 * g + 3] * scale;
            *reinterpret_cast<uint2*>(smem + b_lane * TROW + c0(j, g) * 2) =
                make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
          }
      }
      __syncthreads();
#pragma unroll 4
      for (int e = tid; e < BROWS * PER_ROW; e += THREADS) {
        const int b = e / PER_ROW, ck = e % PER_ROW;
        const int64_t r = m0 + band_row(i, b);
        const int c = n0 + 8 * ck;
        if (r < a.M && c < a.N)
          *reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.C) + r * a.N + c) =
              *reinterpret_cast<const uint4*>(smem + b * TROW + 16 * ck);
      }
      __syncthreads();  // the staged band is read before the next band's addend lands
    }
  } else {
    // Sum of squares of each row: over the lane's columns, then its partner
    // half-wave (lane ^ 32), then the WAVES_N waves of the row band in a
    // fixed order through LDS.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      bias_relu(i);
      float s = 0.0f;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) s = fmaf(acc[i][j][e], acc[i][j][e], s);
      s += __shfl_xor(s, 32);
      if (half == 0) red[wn * BM + a_base_row + i * 32 + row_in_blk] = s;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = a_base_row + i * 32 + row_in_blk;
      float ss = 0.0f;
#pragma unroll
      for (int w = 0; w < C::WAVES_N; ++w) ss += red[w * BM + r];
      store_band(i, ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f);
    }
    flush_tile();
  }
}

// ---------------------------------------------------------------------------
// bf16 GEMM with register-staged loads, for one A source without a row map
// and without the L2 epilogue (the Q transform and the neighbour half of W).
//
// A 256 x 256 tile per block of 4 waves (2 x 2, 128 x 128 each). K runs in
// chunks of 64 columns, i.e. 128 bytes per row: each load instruction of a
// wave reads 8 whole rows of a chunk (8 lanes x 16 B per row), so every
// request is a full 128-byte line. Chunks travel global -> VGPR -> LDS: two
// register buffers keep chunks c + 2 and c + 3 in flight while chunk c is
// multiplied from one LDS stage and chunk c + 1 waits in the other. In a row
// of a stage, 16-byte vector v sits in slot v ^ ((row >> 1) & 7): a 16-byte
// access is served 16 lanes at a time from 64 banks (two 128-byte rows), so
// the 16 lanes that write two rows, and the 16 rows read by a fragment
// instruction's lane group, fall on distinct banks. Missing rows and the K
// tail read zeros through the buffer descriptors' range checks.
// ---------------------------------------------------------------------------
template <int WAVES_M_, int WAVES_N_>
struct RsCfg {
  static constexpr int BM = 256, BN = 256, BK = 64;
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, NW = WAVES_M * WAVES_N;
  static constexpr int THREADS = 64 * NW;
  static constexpr int ROWS = BM + BN;                 // rows of a stage (A rows, then B rows)
  static constexpr int ROW_BYTES = BK * 2;             // 128
  static constexpr int STAGE_BYTES = ROWS * ROW_BYTES; // 64 KB
  static constexpr int RSTEP = THREADS / 8;            // stage rows per block load instruction
  static constexpr int LOADS = ROWS / RSTEP;           // 16-byte vectors per thread per chunk
  static constexpr int SLICE = LOADS / 4;              // loads (and stores) per k-step
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int TM = WM / 32, TN = WN / 32;     // 32 x 32 blocks per wave
  static_assert(LOADS % 4 == 0 && TM * TN >= TM + TN + 2, "k-step interleave pattern");
};

template <typename C>
__global__ __launch_bounds__(C::THREADS) void gemm_rs_kernel(GemmLaunch a) {
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, THREADS = C::THREADS;
  constexpr int ROW_BYTES = C::ROW_BYTES, STAGE_BYTES = C::STAGE_BYTES, RSTEP = C::RSTEP;
  constexpr int LOADS = C::LOADS, SLICE = C::SLICE, TM = C::TM, TN = C::TN;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * STAGE_BYTES + BN * 4];
  float* bias_s = reinterpret_cast<float*>(smem + 2 * STAGE_BYTES);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;

  // Tile coordinates are wave-uniform; readfirstlane keeps them (and the
  // buffer descriptors built from them) in scalar registers.
  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = __builtin_amdgcn_readfirstlane(xcd_tile(blockIdx.x, gridDim.x));
  const int tm = __builtin_amdgcn_readfirstlane(tile / tiles_n);
  const int n0 = __builtin_amdgcn_readfirstlane((tile - tm * tiles_n) * BN);
  const int64_t m0 = (int64_t)tm * BM;
  const int K = a.K0;
  for (int c = tid; c < BN; c += THREADS)
    bias_s[c] = (a.bias && n0 + c < a.N) ? a.bias[n0 + c] : 0.0f;

  // Load slot i of this thread: stage row (tid >> 3) + RSTEP i (A rows for
  // i < LOADS / 2, B rows after), 16-byte vector tid & 7 of the row's chunk.
  // Loads go
  // through buffer descriptors spanning the rows of this tile that exist, so
  // missing rows read zeros; the K tail takes an offset past every
  // descriptor's range (also zeros). No load is behind a branch.
  const int r0 = tid >> 3, v = tid & 7;
  const int64_t a_rows = a.M < a.rows_a0 ? a.M : a.rows_a0;  // rows of A that exist
  const int64_t a_have = a_rows - m0 < 0 ? 0 : (a_rows - m0 > BM ? BM : a_rows - m0);
  const int64_t b_have = a.N - n0 < 0 ? 0 : (a.N - n0 > BN ? BN : a.N - n0);
  const int a_bytes = __builtin_amdgcn_readfirstlane((int)(a_have * a.lda0 * 2));
  const int b_bytes = __builtin_amdgcn_readfirstlane((int)(b_have * a.ldb * 2));
  const __amdgpu_buffer_rsrc_t a_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<unsigned char*>(static_cast<const unsigned char*>(a.A0)) + m0 * a.lda0 * 2,
      (short)0, a_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t b_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<unsigned char*>(static_cast<const unsigned char*>(a.B)) + (int64_t)n0 * a.ldb * 2,
      (short)0, b_bytes, 0x00020000);
  const int a_off0 = r0 * (int)a.lda0 * 2 + v * 16, a_step = RSTEP * (int)a.lda0 * 2;
  const int b_off0 = r0 * (int)a.ldb * 2 + v * 16, b_step = RSTEP * (int)a.ldb * 2;
  const int nchunks = (K + BK - 1) / BK;

  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 stage_regs[2][LOADS];
  auto load_chunk = [&](int chunk, u32x4 (&r)[LOADS]) __attribute__((always_inline)) {
    // Bit 31 set (arithmetically, not by a select) sends the K tail past the
    // descriptors' ranges.
    const int oob = (int)((uint32_t)(K - 1 - (chunk * BK + v * 8)) & 0x80000000u);
    const int koff = chunk * ROW_BYTES;
#pragma unroll
    for (int i = 0; i < LOADS / 2; ++i)
      r[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           a_rsrc, (a_off0 + i * a_step + koff) | oob, 0, 0));
#pragma unroll
    for (int i = 0; i < LOADS / 2; ++i)
      r[LOADS / 2 + i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                       b_rsrc, (b_off0 + i * b_step + koff) | oob,
                                                       0, 0));
  };
  // Quarter q of a chunk: load slots SLICE q .. SLICE (q + 1) - 1 (A rows for q < 2).
  auto load_slice = [&](int chunk, u32x4 (&r)[LOADS], int q) __attribute__((always_inline)) {
    const int oob = (int)((uint32_t)(K - 1 - (chunk * BK + v * 8)) & 0x80000000u);
    const int koff = chunk * ROW_BYTES;
#pragma unroll
    for (int u = 0; u < SLICE; ++u) {
      const int i = SLICE * q + u;
      if (i < LOADS / 2)
        r[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                             a_rsrc, (a_off0 + i * a_step + koff) | oob, 0, 0));
      else
        r[i] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       b_rsrc, (b_off0 + (i - LOADS / 2) * b_step + koff) | oob, 0, 0));
    }
  };
  // ((r0 + RSTEP i) >> 1) & 7 == (r0 >> 1) & 7: one slot for all of this
  // thread's rows.
  const int wslot = (v ^ ((r0 >> 1) & 7)) * 16;
  auto store_chunk = [&](int stage, const u32x4 (&r)[LOADS]) __attribute__((always_inline)) {
    unsigned char* base = smem + stage * STAGE_BYTES + r0 * ROW_BYTES + wslot;
#pragma unroll
    for (int i = 0; i < LOADS; ++i)
      *reinterpret_cast<u32x4*>(base + i * RSTEP * ROW_BYTES) = r[i];
  };
  auto store_slice = [&](int stage, const u32x4 (&r)[LOADS], int q) __attribute__((always_inline)) {
    unsigned char* base = smem + stage * STAGE_BYTES + r0 * ROW_BYTES + wslot;
#pragma unroll
    for (int u = 0; u < SLICE; ++u)
      *reinterpret_cast<u32x4*>(base + (SLICE * q + u) * RSTEP * ROW_BYTES) = r[SLICE * q + u];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  // Fragment reads: lane l takes row (l & 31) of a 32-row block and vector
  // 2 ks + (l >> 5) of k-step ks; rows of a block start at multiples of 8.
  const int frow = lane & 31, half = lane >> 5;
  const int fa = (wm * C::WM + frow) * ROW_BYTES;
  const int fb = (BM + wn * C::WN + frow) * ROW_BYTES;
  struct Frags {
    u32x4 a[TM], b[TN];
  };
  auto read_frags = [&](int stage, int ks, Frags& f) __attribute__((always_inline)) {
    const unsigned char* st = smem + stage * STAGE_BYTES;
    const int slot = ((2 * ks + half) ^ ((frow >> 1) & 7)) * 16;
#pragma unroll
    for (int i = 0; i < TM; ++i)
      f.a[i] = *reinterpret_cast<const u32x4*>(st + fa + i * 32 * ROW_BYTES + slot);
#pragma unroll
    for (int j = 0; j < TN; ++j)
      f.b[j] = *reinterpret_cast<const u32x4*>(st + fb + j * 32 * ROW_BYTES + slot);
  };
  auto mfma = [&](const Frags& f) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, f.b[j]), __builtin_bit_cast(bf16x8, f.a[i]), acc[i][j],
            0, 0, 0);
  };

  // Prologue: chunk 0 into stage 0; chunks 1 and 2 in flight. (The compiler
  // places the vmcnt waits before each store from the loaded registers.)
  load_chunk(0, stage_regs[0]);
  load_chunk(1, stage_regs[1]);
  store_chunk(0, stage_regs[0]);
  load_chunk(2, stage_regs[0]);
  lds_barrier();

  // One chunk: chunk c + 1 (the oldest loads in flight) goes into the other
  // stage, whose last readers passed the barrier that ended the previous
  // step; its registers then take chunk c + 3; chunk c is multiplied. The
  // stage and register-buffer indices are compile-time (two steps per loop
  // trip), so the buffers stay in registers.
  auto step = [&](int c, auto CUR) __attribute__((always_inline)) {
    constexpr int cur = decltype(CUR)::value, nxt = cur ^ 1;
    Frags f[2];
    read_frags(cur, 0, f[0]);
    // Scheduling fences at the k-step boundaries keep each step's fragment
    // reads inside the previous step, so the MFMAs wait only on reads issued
    // a whole k-step earlier (left to itself the scheduler pulled the current
    // step's B reads in between its own MFMAs, exposing their latency).
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      // A quarter of chunk c + 1's LDS writes and of chunk c + 3's loads per
      // k-step, the next k-step's fragment reads, and the 16 MFMAs of this
      // k-step, interleaved one for one so that LDS and memory traffic run
      // under the matrix work.
      if (ks < 3) read_frags(cur, ks + 1, f[(ks + 1) & 1]);
      store_slice(nxt, stage_regs[nxt], ks);
      load_slice(c + 3, stage_regs[nxt], ks);
      mfma(f[ks & 1]);
      constexpr int NR = TM + TN;              // fragment reads of a k-step
      if (ks < 3) {
#pragma unroll
        for (int i = 0; i < NR; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        }
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, NR, 0);
      }
      constexpr int REST = TM * TN - NR;       // MFMAs left for the writes and loads
      constexpr int PER = SLICE < REST / 2 ? 1 : (SLICE + REST / 2 - 1) / (REST / 2);
#pragma unroll
      for (int i = 0; i < SLICE; i += PER) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // MFMA
        __builtin_amdgcn_sched_group_barrier(0x200, PER, 0);  // DS write
      }
#pragma unroll
      for (int i = 0; i < SLICE; i += PER) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, PER, 0);  // VMEM read
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    lds_barrier();
  };
  // An odd chunk count runs one more chunk, read entirely out of range (all
  // zeros), so the loop body has no exit in the middle.
  for (int c = 0; c < nchunks; c += 2) {
    step(c, std::integral_constant<int, 0>{});
    step(c + 1, std::integral_constant<int, 1>{});
  }

  // ---- epilogue: bias (+ ReLU) into a bf16 C tile in LDS, then row stores ---
  // After the last chunk's barrier both stages are free; they hold the
  // 256 x 256 tile, row r at byte 512 r with its 16-byte slot s (8 columns)
  // at position s ^ (r & 31), so the lanes' 4-column pieces (16 rows per LDS
  // pass) and the row runs read back (16 slots of one row per pass) fall on
  // distinct banks. Each row then leaves as 32 x 16 B contiguous stores.
  // Lane l holds output row WM wm + 32 i + (l & 31) of the tile and, for group
  // g of block j, columns WN wn + 32 j + 8 g + 4 (l >> 5) + 0..3.
  static_assert(2 * STAGE_BYTES >= BM * BN * 2 && BN == 256, "C tile fits the two stages");
  constexpr int ROWB = BN * 2;  // bytes per C tile row
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int rt = wm * C::WM + i * 32 + frow;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int cb = wn * C::WN + j * 32 + 8 * g + 4 * half;
        const float4 bv = *reinterpret_cast<const float4*>(bias_s + cb);
        float x0 = acc[i][j][4 * g] + bv.x, x1 = acc[i][j][4 * g + 1] + bv.y;
        float x2 = acc[i][j][4 * g + 2] + bv.z, x3 = acc[i][j][4 * g + 3] + bv.w;
        if (a.relu) {
          x0 = fmaxf(x0, 0.0f);
          x1 = fmaxf(x1, 0.0f);
          x2 = fmaxf(x2, 0.0f);
          x3 = fmaxf(x3, 0.0f);
        }
        const int slot = (cb >> 3) ^ (rt & 31);
        *reinterpret_cast<uint2*>(smem + rt * ROWB + slot * 16 + half * 8) =
            make_uint2(pack_bf16x2(x0, x1), pack_bf16x2(x2, x3));
      }
  }
  __syncthreads();
#pragma unroll 4
  for (int k = 0; k < BM * (BN / 8) / THREADS; ++k) {
    const int e = k * THREADS + tid;
    const int rt = e >> 5, sl = e & 31;
    const int64_t r = m0 + rt;
    const int c = n0 + sl * 8;
    if (r < a.M && c < a.N) {
      // Streaming stores: the output is not read again by this kernel, so it
      // should not push the reused B rows out of L2.
      const uint4 v = *reinterpret_cast<const uint4*>(smem + rt * ROWB + ((sl ^ (rt & 31)) * 16));
      typedef uint32_t u32x4s __attribute__((ext_vector_type(4)));
      __builtin_nontemporal_store(
          __builtin_bit_cast(u32x4s, v),
          reinterpret_cast<u32x4s*>(static_cast<uint16_t*>(a.C) + r * a.N + c));
    }
  }
}

// The register-staged kernel covers bf16 launches with one A source, no row
// map, no addend and no L2 epilogue, and rows whose byte strides keep 16-byte
// vectors aligned.
bool use_rs(const GemmLaunch& a) {
  const int64_t ldb = a.ldb ? a.ldb : a.K0;
  // Buffer offsets are 32-bit: a tile's 256 rows must span < 2^31 bytes.
  // The epilogue writes rows in 8-column (16-byte) pieces: N % 8 == 0.
  return a.bf16 && !a.l2norm && a.K1 == 0 && !a.rowmap && !a.addend && a.K0 % 8 == 0 &&
         a.N % 8 == 0 && a.lda0 % 8 == 0 && ldb % 8 == 0 && a.lda0 <= (1 << 20) &&
         ldb <= (1 << 20) && reinterpret_cast<uintptr_t>(a.A0) % 16 == 0 &&
         reinterpret_cast<uintptr_t>(a.B) % 16 == 0 && reinterpret_cast<uintptr_t>(a.C) % 16 == 0;
}

#ifndef PINSAGE_RS_CFG
#define PINSAGE_RS_CFG RsCfg<2, 2>
#endif
hipError_t launch_rs(GemmLaunch a, hipStream_t s) {
  using C = PINSAGE_RS_CFG;
  if (!a.ldb) a.ldb = a.K0;
  const int64_t tiles = ((a.M + C::BM - 1) / C::BM) * (int64_t)((a.N + C::BN - 1) / C::BN);
  if (tiles <= 0) return hipSuccess;
  if (tiles > 0x7FFFFFFFll) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gemm_rs_kernel<C>, dim3((unsigned)tiles), dim3(C::THREADS), 0, s, a);
  return hipGetLastError();
}

template <typename C>
hipError_t launch_cfg(const GemmLaunch& a, hipStream_t s) {
  const int64_t tiles = ((a.M + C::BM - 1) / C::BM) * (int64_t)((a.N + C::BN - 1) / C::BN);
  if (tiles <= 0) return hipSuccess;
  if (tiles > 0x7FFFFFFFll) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gemm_kernel<C>, dim3((unsigned)tiles), dim3(C::THREADS), 0, s, a);
  return hipGetLastError();
}

// Tile shapes per (dtype, epilogue, output width).
#ifndef PINSAGE_CFG_Q_BF16
#define PINSAGE_CFG_Q_BF16 Cfg<true, 256, 256, 2, 2, false, 4>
#endif
#ifndef PINSAGE_CFG_Q_F32
#define PINSAGE_CFG_Q_F32 Cfg<false, 256, 256, 4, 4, false, 4>
#endif
#ifndef PINSAGE_CFG_W256_BF16
#define PINSAGE_CFG_W256_BF16 Cfg<true, 128, 256, 2, 4, true, 3>
#endif
#ifndef PINSAGE_CFG_W256_F32
#define PINSAGE_CFG_W256_F32 Cfg<false, 128, 256, 2, 4, true, 3>
#endif
#ifndef PINSAGE_CFG_W512_BF16
#define PINSAGE_CFG_W512_BF16 Cfg<true, 128, 512, 2, 4, true, 3>
#endif
#ifndef PINSAGE_CFG_W512_F32
#define PINSAGE_CFG_W512_F32 Cfg<false, 128, 512, 2, 4, true, 3>
#endif

template <bool BF16>
hipError_t launch_typed(const GemmLaunch& a, hipStream_t s) {
  if (!a.l2norm) {  // Q transform and the neighbour half of W share the tiles
    if constexpr (BF16) return launch_cfg<PINSAGE_CFG_Q_BF16>(a, s);
    else return launch_cfg<PINSAGE_CFG_Q_F32>(a, s);
  }
  // The block must span every output column for the fused row norm.
  if (a.N <= 64) return launch_cfg<Cfg<BF16, 128, 64, 4, 1, true, 4>>(a, s);
  if (a.N <= 128) return launch_cfg<Cfg<BF16, 128, 128, 2, 2, true, 4>>(a, s);
  if (a.N <= 256) {
    if constexpr (BF16) return launch_cfg<PINSAGE_CFG_W256_BF16>(a, s);
    else return launch_cfg<PINSAGE_CFG_W256_F32>(a, s);
  }
  if (a.N <= 512) {
    if constexpr (BF16) return launch_cfg<PINSAGE_CFG_W512_BF16>(a, s);
    else return launch_cfg<PINSAGE_CFG_W512_F32>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(const GemmLaunch& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  ProfileScope prof(a.prof_class >= 0 ? a.prof_class : (a.l2norm ? kKGemmW : (a.relu ? kKGemmQ : kKGemmR)), s);
#ifndef PINSAGE_GEMM_NO_RS
  if (use_rs(a)) return launch_rs(a, s);
#endif
  return a.bf16 ? launch_typed<true>(a, s) : launch_typed<false>(a, s);
}

}  // namespace pinsage
