// bf16 GEMM on gfx950 matrix cores, C[M,N] = A[M,K] * B[N,K]^T, fp32 accumulation,
// with the layer's epilogues fused in.
//
// The four projections of the layer (QKV, O, gate/up, down) are the dense
// contractions of the denoising step (the L*d^2 term of the complexity
// equation, Sec. 3.1).  Tiling: 256x256 block tile, K step 64, four waves in
// a 2x2 grid, each wave owning a 128x128 sub-tile as 4x4 tiles of the
// 32x32x16 bf16 MFMA.  Operand tiles move HBM -> LDS with direct-to-LDS
// 16-byte loads into a two-stage ring; the 16-byte chunks of each 128-byte
// LDS row are XOR-swizzled so that the MFMA fragment reads of 16 consecutive
// rows land in distinct banks.
//
// Epilogues:
//   SCALE   C = bf16(acc * rowscale[r])         folded RMSNorm before QKV
//   RESID   C = bf16(R[r,c] + acc)              residual after O and down
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

  const int M = rows_from(p.m_ptr, p.m_ub);
  const int tiles_m = (p.m_ub + BM - 1) / BM;
  const int tiles_n = p.N / BN;
  int tm, tn;
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  if (m0 >= M) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1;
  const int wn = wave & 1;

  // ---- global -> LDS load geometry ---------------------------------------
  // Wave w fills tile rows [64w, 64w+64) of A and of B, eight rows per
  // instruction; lane l of instruction j writes LDS chunk (l & 7) of row
  // 64w + 8j + (l >> 3), which holds logical K-chunk (l & 7) ^ swz(row).
  const uint16_t* A = static_cast<const uint16_t*>(p.A);
  const uint16_t* Bm = static_cast<const uint16_t*>(p.B);
  uint16_t* C = static_cast<uint16_t*>(p.C);
  const uint16_t* R = static_cast<const uint16_t*>(p.R);
  const uint16_t* a_ptr[8];
  const uint16_t* b_ptr[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = wave * 64 + j * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ (lane >> 3) ^ (j & 1);
    int ga = m0 + row;
    ga = ga < M ? ga : M - 1;
    a_ptr[j] = A + (size_t)ga * p.lda + lc * 8;
    b_ptr[j] = Bm + (size_t)(n0 + row) * p.ldb + lc * 8;
  }
  lds_u8_t* lds = (lds_u8_t*)smem;

  auto issue_stage = [&](int stage, int k0) {
    lds_u8_t* sa = lds + stage * STAGE_BYTES + wave * 64 * ROW_BYTES;
    lds_u8_t* sb = sa + BM * ROW_BYTES;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      __builtin_amdgcn_global_load_lds((const glb_void_t*)(a_ptr[j] + k0),
                                       (lds_void_t*)(sa + j * 8 * ROW_BYTES), 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      __builtin_amdgcn_global_load_lds((const glb_void_t*)(b_ptr[j] + k0),
                                       (lds_void_t*)(sb + j * 8 * ROW_BYTES), 16, 0, 0);
    }
  };

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

  const int KT = p.K / BK;
  issue_stage(0, 0);
  for (int kt = 0; kt < KT; ++kt) {
    __syncthreads();  // stage kt landed; stage kt+1 is free
    if (kt + 1 < KT) issue_stage((kt + 1) & 1, (kt + 1) * BK);
    const uint8_t* sa = smem + (kt & 1) * STAGE_BYTES;
    const uint8_t* sb = sa + BM * ROW_BYTES;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int chunk = ((2 * ks + fhalf) ^ fsw) * 16;
      bf16x8_t af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + i * 32 + fr;
        af[i] = as_bf16x8(*reinterpret_cast<const uint4*>(sa + row * ROW_BYTES + chunk));
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = wn * 128 + j * 32 + fr;
        bf[j] = as_bf16x8(*reinterpret_cast<const uint4*>(sb + row * ROW_BYTES + chunk));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  }

  // ---- epilogue -----------------------------------------------------------
  // Accumulator register r of a 32x32 tile holds row 8*(r/4) + 4*(lane/32) + r%4
  // and column lane%32.
  const int row_base = m0 + wm * 128 + fhalf * 4;
  if constexpr (EPI == EPI_SCALE || EPI == EPI_RESID) {
    const int col_base = n0 + wn * 128 + fr;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row_base + i * 32 + (r >> 2) * 8 + (r & 3);
        if (row < M) {
          if constexpr (EPI == EPI_SCALE) {
            const float s = p.rs[row];
#pragma unroll
            for (int j = 0; j < 4; ++j)
              C[(size_t)row * p.ldc + col_base + j * 32] = f2bf(acc[i][j][r] * s);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const size_t c = col_base + j * 32;
              C[(size_t)row * p.ldc + c] = f2bf(bf2f(R[(size_t)row * p.ldr + c]) + acc[i][j][r]);
            }
          }
        }
      }
    }
  } else {
    const int acol_base = (n0 + wn * 128) / 2 + fr;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row_base + i * 32 + (r >> 2) * 8 + (r & 3);
        const bool ok = row < M;
        const float s = ok ? p.rs[row] : 0.0f;
        float a[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const float g = acc[i][2 * q][r] * s;
          const float u = acc[i][2 * q + 1][r] * s;
          a[q] = silu(g) * u;
          if (ok) C[(size_t)row * p.ldc + acol_base + q * 32] = f2bf(a[q]);
        }
        if constexpr (EPI == EPI_SWIGLU_COUNT) {
          const uint64_t m0b = __ballot(fabsf(a[0]) < p.eps);
          const uint64_t m1b = __ballot(fabsf(a[1]) < p.eps);
          if ((lane & 31) == 0 && ok) {
            const int sh = fhalf * 32;
            const int c = __popcll((m0b >> sh) & 0xffffffffull) + __popcll((m1b >> sh) & 0xffffffffull);
            atomicAdd(p.cnt + row, c);
          }
        }
      }
    }
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
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace seer
