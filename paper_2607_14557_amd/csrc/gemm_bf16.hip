// bf16 GEMM on gfx950 matrix cores, C[M,N] = A[M,K] * B[N,K]^T, fp32 accumulation,
// with the layer's epilogues fused in.
//
// The four projections of the layer (QKV, O, gate/up, down) are the dense
// contractions of the denoising step (the L*d^2 term of the complexity
// equation, Sec. 3.1).  Tiling: 256x256 block tile, K step 64, four waves in
// a 2x2 grid, each wave owning a 128x128 sub-tile as 4x4 tiles of the
// 32x32x16 bf16 MFMA.  The next K step's operand tiles are loaded into
// registers while the current one is multiplied out of LDS, then written to
// the other half of a two-stage LDS ring; the 16-byte chunks of each 128-byte
// LDS row are XOR-swizzled so that the MFMA fragment reads of 16 consecutive
// rows land in distinct banks.  Fragments of the next 16-wide K slice are read
// from LDS before the current slice's MFMAs are issued.
//
// Epilogues:
//   SCALE   C = bf16(acc * rowscale[r])         folded RMSNorm before QKV
//   RESID   C = bf16(R[r,c] + acc)              residual add
//   RESID_DUAL  as RESID, plus an fp32 copy     residual after O (h1 kept in fp32)
//   RESID_R32   C = bf16(R32[r,c] + acc)        residual after down, fp32 h1
//   SWIGLU  act = silu(acc_g * s) * (acc_u * s) gate/up with folded RMSNorm;
//           the packed weight interleaves 32 gate rows with 32 up rows, so a
//           wave holds matching gate and up columns in its registers
//   SWIGLU_COUNT  as SWIGLU, plus the per-row count of |act| < eps on the
//           fp32 values (wave ballot + popcount, one atomic per row and wave)
#include "common.h"
#include "kernels.h"

namespace seer {

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;
constexpr int GROUP_M = 8;
constexpr int ROW_BYTES = BK * 2;                   // 128 bytes per tile row
constexpr int STAGE_BYTES = (BM + BN) * ROW_BYTES;  // 64 KiB

__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Block id -> (tile_m, tile_n).  Consecutive workgroup ids are spread round
// robin over the 8 XCDs; re-number so that each XCD walks a contiguous range
// of logical tiles, then raster those in groups of GROUP_M tile rows so the
// blocks resident on one XCD share A row-tiles and B column-tiles in its L2.
__device__ __forceinline__ void tile_of(int bid, int nblk, int tiles_m, int tiles_n,
                                        int& tm, int& tn) {
  const int per = nblk >> 3;
  int lid = bid;
  if (bid < (per << 3)) lid = (bid & 7) * per + (bid >> 3);
  const int gsz = GROUP_M * tiles_n;
  const int g = lid / gsz;
  const int first_m = g * GROUP_M;
  int gm = tiles_m - first_m;
  gm = gm < GROUP_M ? gm : GROUP_M;
  const int in = lid - g * gsz;
  tm = first_m + in % gm;
  tn = in / gm;
}

}  // namespace

template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * STAGE_BYTES];

  // Tile geometry follows the real row count read on the device, so that the
  // blocks carrying work are spread over every XCD; surplus blocks of the
  // upper-bound grid exit at once.
  const int M = rows_from(p.m_ptr, p.m_ub);
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = p.N / BN;
  const int ntiles = tiles_m * tiles_n;
  if ((int)blockIdx.x >= ntiles) return;
  int tm, tn;
  tile_of(blockIdx.x, ntiles, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM;
  const int n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1;
  const int wn = wave & 1;

  uint16_t* C = static_cast<uint16_t*>(p.C);
  const uint16_t* R = static_cast<const uint16_t*>(p.R);

  // ---- global -> register -> LDS staging -----------------------------------
  // Thread t moves 16-byte chunks c = t + 256 i (i < 8) of each 256x64 operand
  // tile: tile row c / 8, K-chunk c % 8 -- eight consecutive threads read one
  // 128-byte row segment.  In LDS the chunk lands at position chunk ^ swz(row).
  const int srow = tid >> 3;          // + 32 i
  const int schunk = tid & 7;
  // 32-bit byte offsets from the uniform bases (operands are < 4 GiB); rows of
  // A past M re-read row M-1 (never stored).  swz(row) is the same for
  // row = srow + 32 i, so the LDS slot is one base plus an immediate.
  const char* Ab = static_cast<const char*>(p.A);
  const char* Bb = static_cast<const char*>(p.B);
  uint32_t a_off[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int ga = m0 + srow + 32 * i;
    ga = ga < M ? ga : M - 1;
    a_off[i] = (uint32_t)ga * (uint32_t)p.lda * 2u + (uint32_t)schunk * 16u;
  }
  const uint32_t b_off = (uint32_t)(n0 + srow) * (uint32_t)p.ldb * 2u + (uint32_t)schunk * 16u;
  const uint32_t b_step = 32u * (uint32_t)p.ldb * 2u;
  const int s_off = srow * ROW_BYTES + ((schunk ^ swz(srow)) << 4);
  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Fragment read geometry: lane l reads row (l & 31) of a 32-row MFMA tile
  // and the 16-byte K-chunk 2*ks + (l >> 5).
  const int fr = lane & 31;
  const int fsw = swz(fr);
  const int fhalf = lane >> 5;
  const int a_row0 = (wm * 128 + fr) * ROW_BYTES;
  const int b_row0 = BM * ROW_BYTES + (wn * 128 + fr) * ROW_BYTES;

  // Software pipeline, two K tiles of look-ahead: while tile t is multiplied
  // out of LDS stage t%2, tile t+1 (loaded into registers one iteration
  // earlier) is written into stage (t+1)%2 between the MFMAs, and the loads of
  // tile t+2 are in flight.  Two register sets alternate, so the loop is
  // unrolled by two; K/64 is even for every shape the bf16 path accepts.
  u32x4_t ra0[8], rb0[8], ra1[8], rb1[8];
  bf16x8_t af[2][4], bfr[2][4];
  const int KT = p.K / BK;

#define SEER_GLOAD(RA, RB, T, P)                                                    \
  {                                                                                 \
    const int t_ = (T) < KT ? (T) : KT - 1;                                         \
    const char* ak_ = Ab + (size_t)t_ * (BK * 2);                                   \
    const char* bk_ = Bb + (size_t)t_ * (BK * 2);                                   \
    _Pragma("unroll") for (int i = 2 * (P); i < 2 * (P) + 2; ++i) {                 \
      RA[i] = *reinterpret_cast<const u32x4_t*>(ak_ + a_off[i]);                    \
      RB[i] = *reinterpret_cast<const u32x4_t*>(bk_ + b_off + i * b_step);          \
    }                                                                               \
  }
#define SEER_LSTORE2(RA, RB, STG, I0)                                               \
  {                                                                                 \
    uint8_t* sa_ = smem + (STG) * STAGE_BYTES + s_off;                              \
    *reinterpret_cast<u32x4_t*>(sa_ + ((I0) + 0) * 32 * ROW_BYTES) = RA[(I0) + 0];  \
    *reinterpret_cast<u32x4_t*>(sa_ + ((I0) + 1) * 32 * ROW_BYTES) = RA[(I0) + 1];  \
    *reinterpret_cast<u32x4_t*>(sa_ + (BM + ((I0) + 0) * 32) * ROW_BYTES) = RB[(I0) + 0];  \
    *reinterpret_cast<u32x4_t*>(sa_ + (BM + ((I0) + 1) * 32) * ROW_BYTES) = RB[(I0) + 1];  \
  }
#define SEER_FLOAD(ST, KS, BUF)                                                     \
  {                                                                                 \
    const int chunk_ = ((2 * (KS) + fhalf) ^ fsw) << 4;                             \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                 \
      af[BUF][i] = __builtin_bit_cast(bf16x8_t,                                     \
          *reinterpret_cast<const u32x4_t*>((ST) + a_row0 + i * 32 * ROW_BYTES + chunk_)); \
      bfr[BUF][i] = __builtin_bit_cast(bf16x8_t,                                    \
          *reinterpret_cast<const u32x4_t*>((ST) + b_row0 + i * 32 * ROW_BYTES + chunk_)); \
    }                                                                               \
  }
  // One K tile of 4 slices x 16 MFMAs.  Each slice is its own scheduling
  // region (sched_barrier fences), holding: the 8 fragment reads of the next
  // slice, issued first and paired with the first MFMAs so they have the whole
  // slice to land; 4 global loads of tile T+2; 4 LDS writes of tile T+1.  Slice
  // 0's own fragments are read in a region of their own at the top.
#define SEER_TILE(T, RA, RB, RN, RNB)                                               \
  {                                                                                 \
    const uint8_t* st_ = smem + ((T) & 1) * STAGE_BYTES;                            \
    SEER_FLOAD(st_, 0, 0);                                                          \
    __builtin_amdgcn_sched_barrier(0);                                              \
    _Pragma("unroll") for (int ks = 0; ks < 4; ++ks) {                              \
      const int cur = ks & 1;                                                       \
      if (ks + 1 < 4) SEER_FLOAD(st_, ks + 1, cur ^ 1);                             \
      SEER_GLOAD(RN, RNB, (T) + 2, ks);                                             \
      _Pragma("unroll") for (int i = 0; i < 4; ++i)                                 \
        _Pragma("unroll") for (int j = 0; j < 4; ++j)                               \
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0); \
      SEER_LSTORE2(RA, RB, ((T) + 1) & 1, 2 * ks);                                  \
      if (ks + 1 < 4) {                                                             \
        _Pragma("unroll") for (int g = 0; g < 4; ++g) {                             \
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);                        \
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                        \
        }                                                                           \
      } else {                                                                      \
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);                          \
      }                                                                             \
      _Pragma("unroll") for (int g = 0; g < 4; ++g) {                               \
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                          \
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                          \
      }                                                                             \
      _Pragma("unroll") for (int g = 0; g < 4; ++g) {                               \
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);                          \
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                          \
      }                                                                             \
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);                            \
      __builtin_amdgcn_sched_barrier(0);                                            \
    }                                                                               \
  }

  // prologue: tile 0 -> stage 0, tile 1 in registers (set 1); tile 2 is loaded
  // into set 0 by the slices of tile 0
#pragma unroll
  for (int q = 0; q < 4; ++q) SEER_GLOAD(ra0, rb0, 0, q);
#pragma unroll
  for (int q = 0; q < 4; ++q) SEER_GLOAD(ra1, rb1, 1, q);
  {
    uint8_t* sa_ = smem + s_off;
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4_t*>(sa_ + i * 32 * ROW_BYTES) = ra0[i];
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4_t*>(sa_ + (BM + i * 32) * ROW_BYTES) = rb0[i];
  }
  __syncthreads();
  for (int kt = 0; kt < KT; kt += 2) {
    SEER_TILE(kt, ra1, rb1, ra0, rb0);
    __syncthreads();
    SEER_TILE(kt + 1, ra0, rb0, ra1, rb1);
    __syncthreads();
  }
#undef SEER_GLOAD
#undef SEER_LSTORE2
#undef SEER_FLOAD
#undef SEER_TILE

  // ---- epilogue -----------------------------------------------------------
  // Accumulator register r of a 32x32 tile holds row 8*(r/4) + 4*(lane/32) + r%4
  // and column lane%32.  Each wave stages one 32-row slab of its 128x128 tile
  // at a time through a private LDS region (fp32, padded pitch), then every
  // lane moves 8 consecutive outputs of a row: residual loads and bf16 / fp32
  // stores are 16-byte vector accesses, 16 lanes per 256-byte row segment.
  // For SWIGLU the gate/up pairs are combined in registers first (and the
  // near-zero count taken there), so the slab holds 64 activation columns.
  constexpr int EP = 132;                       // slab pitch in floats
  constexpr bool kGlu = (EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_COUNT);
  constexpr int SC = kGlu ? 64 : 128;           // slab columns
  float* slab = reinterpret_cast<float*>(smem) + wave * (32 * EP);
  const int row_w = m0 + wm * 128;              // first row of the wave tile
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // -- registers -> slab
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = (r >> 2) * 8 + fhalf * 4 + (r & 3);
      if constexpr (kGlu) {
        const int row = row_w + i * 32 + lr;
        const bool ok = row < M;
        const float sc = ok ? p.rs[row] : 0.0f;
        const float av0 = silu(acc[i][0][r] * sc) * (acc[i][1][r] * sc);
        const float av1 = silu(acc[i][2][r] * sc) * (acc[i][3][r] * sc);
        slab[lr * EP + fr] = av0;
        slab[lr * EP + 32 + fr] = av1;
        if constexpr (EPI == EPI_SWIGLU_COUNT) {
          const uint64_t m0b = __ballot(fabsf(av0) < p.eps);
          const uint64_t m1b = __ballot(fabsf(av1) < p.eps);
          if ((lane & 31) == 0 && ok) {
            const int sh = fhalf * 32;
            const int c = __popcll((m0b >> sh) & 0xffffffffull) + __popcll((m1b >> sh) & 0xffffffffull);
            atomicAdd(p.cnt + row, c);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) slab[lr * EP + j * 32 + fr] = acc[i][j][r];
      }
    }
    __syncthreads();
    // -- slab -> global, 8 consecutive outputs per lane
    constexpr int CPR = SC / 8;                 // 8-wide chunks per row
    constexpr int ITERS = 32 * CPR / 64;
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * 64 + lane;
      const int lr = c / CPR;
      const int c8 = (c % CPR) * 8;
      const int row = row_w + i * 32 + lr;
      if (row < M) {
        const float* src = slab + lr * EP + c8;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = src[e];
        if constexpr (kGlu) {
          const size_t o = (size_t)row * p.ldc + (n0 + wn * 128) / 2 + c8;
          u32x4_t pk;
#pragma unroll
          for (int e = 0; e < 4; ++e) pk[e] = pack_bf2(v[2 * e], v[2 * e + 1]);
          *reinterpret_cast<u32x4_t*>(C + o) = pk;
        } else {
          const int col = n0 + wn * 128 + c8;
          const size_t o = (size_t)row * p.ldc + col;
          if constexpr (EPI == EPI_SCALE) {
            const float sc = p.rs[row];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] *= sc;
          } else if constexpr (EPI == EPI_RESID || EPI == EPI_RESID_DUAL) {
            const u32x4_t rv = *reinterpret_cast<const u32x4_t*>(R + (size_t)row * p.ldr + col);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[2 * e] += __uint_as_float(rv[e] << 16);
              v[2 * e + 1] += __uint_as_float(rv[e] & 0xffff0000u);
            }
          } else {
            const f32x4_t* r32 = reinterpret_cast<const f32x4_t*>(p.R32 + (size_t)row * p.ldr + col);
            const f32x4_t r0 = r32[0], r1 = r32[1];
#pragma unroll
            for (int e = 0; e < 4; ++e) { v[e] += r0[e]; v[4 + e] += r1[e]; }
          }
          u32x4_t pk;
#pragma unroll
          for (int e = 0; e < 4; ++e) pk[e] = pack_bf2(v[2 * e], v[2 * e + 1]);
          *reinterpret_cast<u32x4_t*>(C + o) = pk;
          if constexpr (EPI == EPI_RESID_DUAL) {
            f32x4_t* c2 = reinterpret_cast<f32x4_t*>(static_cast<float*>(p.C2) + o);
            c2[0] = f32x4_t{v[0], v[1], v[2], v[3]};
            c2[1] = f32x4_t{v[4], v[5], v[6], v[7]};
          }
        }
      }
    }
    __syncthreads();
  }
}

int launch_gemm_bf16(int epi, const GemmParams& p, hipStream_t s) {
  const int tiles_m = (p.m_ub + BM - 1) / BM;
  const int tiles_n = p.N / BN;
  dim3 grid(tiles_m * tiles_n), block(NT);
  switch (epi) {
    case EPI_SCALE: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SCALE>, grid, block, 0, s, p); break;
    case EPI_RESID: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID>, grid, block, 0, s, p); break;
    case EPI_SWIGLU: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU>, grid, block, 0, s, p); break;
    case EPI_SWIGLU_COUNT:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU_COUNT>, grid, block, 0, s, p); break;
    case EPI_RESID_DUAL:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID_DUAL>, grid, block, 0, s, p); break;
    case EPI_RESID_R32:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID_R32>, grid, block, 0, s, p); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace seer
