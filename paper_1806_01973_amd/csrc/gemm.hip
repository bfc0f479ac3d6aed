// Dense layers of CONVOLVE on gfx950 matrix cores (Algorithm 1):
//   line 1 over every pin once (Sec. 3.4):  P = ReLU(H Q^T + q)
//   lines 2-3:  h' = normalize(ReLU([h_self | n] W^T + w))
// as one templated MFMA GEMM  C = epi(A B^T + bias), A [M x K] assembled from
// two row sources (self rows through an optional row map, then the pooled
// rows), B [N x K] row-major (the PyTorch Linear layout of Q and W).
//
// Work split: a 256-thread block (4 waves) owns a BM x BN output tile; waves
// form a WAVES_M x WAVES_N grid and each wave owns (BM/WAVES_M) x
// (BN/WAVES_N), i.e. TM x TN blocks of 32 x 32. K runs in chunks of BK: the
// next chunk's global 16-byte vectors are loaded into registers while the
// current chunk is multiplied out of LDS. Tiles are stored K-contiguous in
// LDS with a 16-byte row pad so each lane's fragment read is one conflict-free
// 16-byte LDS read.
//
// fp32 storage: v_mfma_f32_32x32x2_f32; the 2 k-values of one MFMA step come
// from the two half-waves, and step j of a chunk pairs half h with chunk
// column h*(BK/2) + j, so each lane reads BK/2 consecutive values of its row.
// bf16 storage: v_mfma_f32_32x32x16_bf16 (gfx950); half h supplies chunk
// columns 16*j + 8*h .. +7. Accumulation is fp32 in both cases.
//
// Epilogue: + bias, ReLU, store in the storage dtype; with L2 the block spans
// all N columns, row sums of squares are reduced across lanes with a fixed
// butterfly and across waves in a fixed order through LDS, and every row is
// scaled by 1/||z|| (zero rows stay zero).
//
// Tile order is XCD-aware: hardware hands block b to XCD b % 8; blocks are
// renumbered so that each XCD gets a contiguous run of tiles, keeping the
// column tiles of one row block on one XCD's L2.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <bool BF16, int BM_, int BN_, int WAVES_M_, int WAVES_N_, bool L2_, int BK_ = 32,
          bool PREFETCH_ = true>
struct Cfg {
  static constexpr bool kBf16 = BF16;
  static constexpr bool kPrefetch = PREFETCH_;  // read next k-step fragments early
  static constexpr bool kTwoSources = L2_;  // the W layer reads [h_self | n]
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
  static constexpr int THREADS = 64 * WAVES_M * WAVES_N;
  static constexpr bool L2 = L2_;
  static constexpr int ESZ = BF16 ? 2 : 4;      // bytes per element
  static constexpr int VEC = 16 / ESZ;           // elements per 16-byte vector
  static constexpr int BK = BK_;                 // K chunk (elements)
  static constexpr int LDK = BK + VEC;           // LDS row stride (elements)
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int VROW = BK / VEC;          // 16-byte vectors per chunk row
  static constexpr int A_VECS = BM * VROW / THREADS;  // per thread
  static constexpr int B_VECS = BN * VROW / THREADS;
  static constexpr int RSTEP = THREADS / VROW;        // rows between a thread's vectors
  static constexpr int STAGE_BYTES = (BM + BN) * LDK * ESZ;
  static constexpr int RED_BYTES = L2 ? WAVES_N * BM * 4 : 0;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile is a multiple of 32x32");
  static_assert((BM * VROW) % THREADS == 0 && (BN * VROW) % THREADS == 0, "even vector split");
  static_assert(THREADS % VROW == 0, "a thread keeps one K offset");
  static_assert(2 * STAGE_BYTES + RED_BYTES <= 160 * 1024, "LDS budget of one workgroup");
};

__device__ __forceinline__ int xcd_tile(int b, int nt) {
  const int per = nt / 8, rem = nt % 8;
  const int xcd = b % 8, slot = b / 8;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

template <typename C>
__global__ __launch_bounds__(C::THREADS) void gemm_kernel(GemmLaunch a) {
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, LDK = C::LDK, VEC = C::VEC;
  constexpr int TM = C::TM, TN = C::TN, VROW = C::VROW, THREADS = C::THREADS;
  constexpr int ESZ = C::ESZ;
  // LDS: two stages of (A tile, B tile), K-contiguous padded rows, then the
  // cross-wave row-norm partials.
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * C::STAGE_BYTES + C::RED_BYTES];
  float* red = reinterpret_cast<float*>(smem + 2 * C::STAGE_BYTES);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int64_t m0 = (int64_t)(tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;
  const int K = a.K0 + a.K1;

  // ---- per-thread load slots (fixed across the K loop) -------------------
  // Thread t loads the 16-byte vector (row r0 + i*RSTEP, column kv) of each
  // chunk, i < A_VECS (resp. B_VECS).
  const int r0 = tid / VROW;
  const int kv = (tid % VROW) * VEC;
  const unsigned char* a0_row[C::A_VECS];
  const unsigned char* a1_row[C::kTwoSources ? C::A_VECS : 1];
#pragma unroll
  for (int i = 0; i < C::A_VECS; ++i) {
    const int64_t gr = m0 + r0 + i * C::RSTEP;
    a0_row[i] = nullptr;
    if constexpr (C::kTwoSources) a1_row[i] = nullptr;
    if (gr < a.M) {
      const int64_t src = a.rowmap ? (int64_t)a.rowmap[gr] : gr;
      if (src >= 0 && src < a.rows_a0)
        a0_row[i] = static_cast<const unsigned char*>(a.A0) + src * a.lda0 * ESZ;
      if constexpr (C::kTwoSources)
        a1_row[i] = static_cast<const unsigned char*>(a.A1) + gr * a.lda1 * ESZ;
    }
  }
  const unsigned char* b_row[C::B_VECS];
#pragma unroll
  for (int i = 0; i < C::B_VECS; ++i) {
    const int r = r0 + i * C::RSTEP;
    b_row[i] = (n0 + r < a.N)
                   ? static_cast<const unsigned char*>(a.B) + (int64_t)(n0 + r) * K * ESZ
                   : nullptr;
  }

  uint4 a_stage[C::A_VECS], b_stage[C::B_VECS];
  auto load_chunk = [&](int kc) {
    const int kk = kc + kv;
#pragma unroll
    for (int i = 0; i < C::A_VECS; ++i) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (kk < a.K0) {
        if (a0_row[i]) v = *reinterpret_cast<const uint4*>(a0_row[i] + (int64_t)kk * ESZ);
      } else if constexpr (C::kTwoSources) {
        if (kk < K && a1_row[i])
          v = *reinterpret_cast<const uint4*>(a1_row[i] + (int64_t)(kk - a.K0) * ESZ);
      }
      a_stage[i] = v;
    }
#pragma unroll
    for (int i = 0; i < C::B_VECS; ++i) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (b_row[i] && kk < K) v = *reinterpret_cast<const uint4*>(b_row[i] + (int64_t)kk * ESZ);
      b_stage[i] = v;
    }
  };
  auto store_chunk = [&](unsigned char* stage) {
    unsigned char* As = stage + (r0 * LDK + kv) * ESZ;
    unsigned char* Bs = stage + (BM * LDK + r0 * LDK + kv) * ESZ;
#pragma unroll
    for (int i = 0; i < C::A_VECS; ++i)
      *reinterpret_cast<uint4*>(As + i * C::RSTEP * LDK * ESZ) = a_stage[i];
#pragma unroll
    for (int i = 0; i < C::B_VECS; ++i)
      *reinterpret_cast<uint4*>(Bs + i * C::RSTEP * LDK * ESZ) = b_stage[i];
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

  // Multiplies one LDS stage into the accumulators; the fragments of the
  // next k-step are read while the current MFMAs issue.
  auto compute = [&](const unsigned char* stage) {
    const unsigned char* As = stage;
    const unsigned char* Bs = stage + BM * LDK * ESZ;
    if constexpr (!C::kBf16) {
      // Half h covers chunk columns [h*BK/2, (h+1)*BK/2), read 8 at a time.
      constexpr int GROUPS = (BK / 2) / 8;
      constexpr int NB = C::kPrefetch ? 2 : 1;
      float fa[NB][TM][8], fb[NB][TN][8];
      auto load = [&](int g, float (&xa)[TM][8], float (&xb)[TN][8]) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const float* p = reinterpret_cast<const float*>(As) +
                           (a_base_row + i * 32 + row_in_blk) * LDK + half * (BK / 2) + 8 * g;
          const float4 x = *reinterpret_cast<const float4*>(p);
          const float4 y = *reinterpret_cast<const float4*>(p + 4);
          xa[i][0] = x.x; xa[i][1] = x.y; xa[i][2] = x.z; xa[i][3] = x.w;
          xa[i][4] = y.x; xa[i][5] = y.y; xa[i][6] = y.z; xa[i][7] = y.w;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const float* p = reinterpret_cast<const float*>(Bs) +
                           (b_base_row + j * 32 + row_in_blk) * LDK + half * (BK / 2) + 8 * g;
          const float4 x = *reinterpret_cast<const float4*>(p);
          const float4 y = *reinterpret_cast<const float4*>(p + 4);
          xb[j][0] = x.x; xb[j][1] = x.y; xb[j][2] = x.z; xb[j][3] = x.w;
          xb[j][4] = y.x; xb[j][5] = y.y; xb[j][6] = y.z; xb[j][7] = y.w;
        }
      };
      if constexpr (C::kPrefetch) load(0, fa[0], fb[0]);
#pragma unroll
      for (int g = 0; g < GROUPS; ++g) {
        const int cb = C::kPrefetch ? (g & 1) : 0;
        if constexpr (C::kPrefetch) {
          if (g + 1 < GROUPS) load(g + 1, fa[(g + 1) & 1], fb[(g + 1) & 1]);
        } else {
          load(g, fa[0], fb[0]);
        }
#pragma unroll
        for (int st = 0; st < 8; ++st)
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[cb][i][st], fb[cb][j][st],
                                                               acc[i][j], 0, 0, 0);
      }
    } else {
      constexpr int KSTEPS = BK / 16;
      constexpr int NB = C::kPrefetch ? 2 : 1;
      bf16x8 fa[NB][TM], fb[NB][TN];
      auto load = [&](int ks, bf16x8 (&xa)[TM], bf16x8 (&xb)[TN]) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
          xa[i] = *reinterpret_cast<const bf16x8*>(
              As + ((a_base_row + i * 32 + row_in_blk) * LDK + 16 * ks + half * 8) * 2);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          xb[j] = *reinterpret_cast<const bf16x8*>(
              Bs + ((b_base_row + j * 32 + row_in_blk) * LDK + 16 * ks + half * 8) * 2);
      };
      if constexpr (C::kPrefetch) load(0, fa[0], fb[0]);
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        const int cb = C::kPrefetch ? (ks & 1) : 0;
        if constexpr (C::kPrefetch) {
          if (ks + 1 < KSTEPS) load(ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
        } else {
          load(ks, fa[0], fb[0]);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cb][i], fb[cb][j], acc[i][j],
                                                                0, 0, 0);
      }
    }
  };

  // Double-buffered K loop: one barrier per chunk; the next chunk's global
  // loads are in flight while the current stage is multiplied out.
  const int nchunks = (K + BK - 1) / BK;
  load_chunk(0);
  store_chunk(smem);
  __syncthreads();
  for (int it = 0; it < nchunks; ++it) {
    const unsigned char* cur = smem + (it & 1) * C::STAGE_BYTES;
    unsigned char* nxt = smem + ((it + 1) & 1) * C::STAGE_BYTES;
    const bool more = it + 1 < nchunks;
    if (more) load_chunk((it + 1) * BK);
    compute(cur);
    if (more) store_chunk(nxt);
    __syncthreads();
  }

  // ---- epilogue -----------------------------------------------------------
  // 32x32 accumulator layout: element e of lane l is row 8*(e/4) + 4*(l/32) +
  // e%4, column l%32 of the block.
  float bias_v[TN];
  int col_of[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    col_of[j] = n0 + b_base_row + j * 32 + row_in_blk;
    bias_v[j] = col_of[j] < a.N ? a.bias[col_of[j]] : 0.0f;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float z = acc[i][j][e] + bias_v[j];
        acc[i][j][e] = (z > 0.0f && col_of[j] < a.N) ? z : 0.0f;
      }

  if constexpr (C::L2) {
    // Row partial sums over this wave's columns.
    float part[TM][16];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float s = 0.0f;
#pragma unroll
        for (int j = 0; j < TN; ++j) s = fmaf(acc[i][j][e], acc[i][j][e], s);
#pragma unroll
        for (int o = 16; o >= 1; o >>= 1) s += __shfl_xor(s, o);
        part[i][e] = s;
      }
    if (row_in_blk == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = a_base_row + i * 32 + 8 * (e / 4) + 4 * half + (e % 4);
          red[wn * BM + r] = part[i][e];
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = a_base_row + i * 32 + 8 * (e / 4) + 4 * half + (e % 4);
        float ss = 0.0f;
#pragma unroll
        for (int w = 0; w < C::WAVES_N; ++w) ss += red[w * BM + r];
        const float inv = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j][e] *= inv;
      }
  }

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t r = m0 + a_base_row + i * 32 + 8 * (e / 4) + 4 * half + (e % 4);
      if (r >= a.M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        if (col_of[j] >= a.N) continue;
        const int64_t o = r * a.N + col_of[j];
        if constexpr (C::kBf16) static_cast<uint16_t*>(a.C)[o] = f32_to_bf16(acc[i][j][e]);
        else static_cast<float*>(a.C)[o] = acc[i][j][e];
      }
    }
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
#define PINSAGE_CFG_Q_BF16 Cfg<true, 128, 128, 2, 2, false, 32>
#endif
#ifndef PINSAGE_CFG_Q_F32
#define PINSAGE_CFG_Q_F32 Cfg<false, 256, 256, 4, 4, false, 16>
#endif
#ifndef PINSAGE_CFG_W256_BF16
#define PINSAGE_CFG_W256_BF16 Cfg<true, 256, 256, 4, 4, true, 32, false>
#endif
#ifndef PINSAGE_CFG_W256_F32
#define PINSAGE_CFG_W256_F32 Cfg<false, 256, 256, 4, 4, true, 32>
#endif
#ifndef PINSAGE_CFG_W512_BF16
#define PINSAGE_CFG_W512_BF16 Cfg<true, 128, 512, 2, 4, true, 32>
#endif
#ifndef PINSAGE_CFG_W512_F32
#define PINSAGE_CFG_W512_F32 Cfg<false, 128, 512, 2, 4, true, 16>
#endif

template <bool BF16>
hipError_t launch_typed(const GemmLaunch& a, hipStream_t s) {
  if (!a.l2norm) {
    if constexpr (BF16) return launch_cfg<PINSAGE_CFG_Q_BF16>(a, s);
    else return launch_cfg<PINSAGE_CFG_Q_F32>(a, s);
  }
  // The block must span every output column for the fused row norm.
  if (a.N <= 64) return launch_cfg<Cfg<BF16, 128, 64, 4, 1, true, 32>>(a, s);
  if (a.N <= 128) return launch_cfg<Cfg<BF16, 128, 128, 2, 2, true, 32>>(a, s);
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
  ProfileScope prof(a.l2norm ? kKGemmW : kKGemmQ, s);
  return a.bf16 ? launch_typed<true>(a, s) : launch_typed<false>(a, s);
}

}  // namespace pinsage
