// bf16 GEMM on gfx950 matrix cores, C[M,N] = A[M,K] * B[N,K]^T, fp32 accumulation,
// with the layer's epilogues fused in.
//
// The four projections of the layer (QKV, O, gate/up, down) are the dense
// contractions of the denoising step (the L*d^2 term of the complexity
// equation, Sec. 3.1).  Tiling: 256x256 block tile, K step 64, four waves side
// by side, each owning all 256 rows and 64 columns of the tile as 8x2 tiles of
// the 32x32x16 bf16 MFMA.
//
// Operands take two different routes:
//   A (activations, shared by all four waves) goes straight from global memory
//     into a four-stage LDS ring with direct-to-LDS buffer loads (1 KiB per
//     instruction, no staging registers), three K tiles ahead; each lane
//     fetches the 16-byte chunk that the XOR swizzle puts at its LDS position,
//     so the fragment reads of 16 consecutive rows land in distinct banks;
//     the four stages are separate arrays and one bare barrier per K tile
//     publishes the next stage;
//   B (weights, 64 columns private to each wave) never touches LDS: the weight
//     prepack stores it fragment-major (frag_b_index), so every operand of a
//     wave is one coalesced 1 KiB load straight into the MFMA registers, issued
//     one K tile ahead.
// Every 16-wide K slice is its own scheduling region in which the next slice's
// A fragments are read first, so LDS latency hides behind a whole slice of
// MFMAs.
//
// Epilogues:
//   SCALE   C = bf16(acc * rowscale[r])         folded RMSNorm before QKV;
//           column tiles from f16_col0 on (V) are stored as fp16 instead;
//           columns below perm_col1 come from the head-permuted q/k rows of
//           the packed weight and are stored back in head order
//   SCALE_ROPE  as SCALE, and the columns below rope_col1 are rotated
//           (rotary embedding of q and k) on the way
//   RESID   C = bf16(R[r,c] + acc)              residual add (the layer uses the
//           two forms below; this one is not launched by the bf16 path)
//   RESID_SPLIT v = R[r,c] + acc: C = bf16(v) and residual after O: h1 as a bf16
//               C2 = bf16(v - C)                high/low pair, exact to ~2^-17
//   RESID_PAIR  C = bf16(R + R2 + acc)          residual after down from that pair
//   SWIGLU  act = silu(acc_g * s) * (acc_u * s) gate/up with folded RMSNorm;
//           the packed weight interleaves 32 gate rows with 32 up rows, so a
//           wave holds matching gate and up columns in its registers
//   SWIGLU_COUNT  as SWIGLU, plus the per-row count of |act| < eps on the
//           fp32 values (per-lane tally, one atomic per row and wave)
//   ARGMAX  per row and 64-column group {max, sum exp(v - max), first argmax}
//           of acc * rowscale (LM head)
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace seer {

namespace {

constexpr int BK = 64;
constexpr int NT = 256;
constexpr int GROUP_M = 4;
constexpr int ROW_BYTES = BK * 2;                   // 128 bytes per A tile row

__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Tiles in the logical order of xcd_remap are laid out by raster in groups of
// GROUP_M tile rows, so the blocks resident on one XCD share A row-tiles and
// B column-tiles in its L2.

__device__ __forceinline__ void raster(int lid, int tiles_m, int tiles_n, int& tm, int& tn) {
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

// s_waitcnt immediate (gfx9 encoding) for vmcnt(vm), lgkmcnt(lgkm), expcnt
// unconstrained.
constexpr int waitcnt_imm(int vm, int lgkm) { return ((vm >> 4) << 14) | (lgkm << 8) | (7 << 4) | (vm & 15); }

// Instruction order inside one K slice of a BMT-row tile (masks: 0x008 MFMA,
// 0x020 VMEM, 0x100 LDS read).  Per slice: the next slice's BMT/32 fragment
// reads, paired two to an MFMA; the loads (BMT/128 of A tile t+3 into LDS,
// two of B tile t+1 into registers), one per MFMA; then the remaining MFMAs.
template <int BMT>
__device__ __forceinline__ void seer_slice_schedule() {
  constexpr int NR = BMT / 32;
  constexpr int NV = BMT / 128 + 2;
  constexpr int NM = 2 * NR;
#pragma unroll
  for (int g = 0; g < NR / 2; ++g) {
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
#pragma unroll
  for (int g = 0; g < NV; ++g) {
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, NM - NR / 2 - NV, 0);
}

// One BMTx256 output tile over K tiles [kt0, kt0 + KT) of 64.  BMT = 256 is
// the main tile; BMT = 128 serves the halves of the tiles of a partly filled
// last round.  Wave w owns columns n0 + 64 w .. +63 and all BMT rows.  PART:
// the tile is split `split` of a K-split launch, and its fp32 sums go to the
// partial scratch instead of through the epilogue.
template <int EPI, int BMT, bool PART = false>
__device__ __forceinline__ void gemm_tile(const GemmParams& p, uint8_t* st0, uint8_t* st1, uint8_t* st2, uint8_t* st3,
                                          int M, int m0, int n0, int kt0, int KT, int split = 0) {
  constexpr int NI = BMT / 32;                      // 32-row MFMA tiles per wave
  constexpr int NA = BMT / 32;                      // A loads (1 KiB each) per wave and K tile
  constexpr int AP = NA / 4;                        // ... per slice

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wcol = n0 + 64 * wave;                  // first (packed) column of the wave

  uint16_t* C = static_cast<uint16_t*>(p.C);
  const uint16_t* R = static_cast<const uint16_t*>(p.R);

  // ---- A: straight into a four-stage LDS ring -----------------------------
  // buffer_load ... lds moves 64 x 16 bytes into 1 KiB of consecutive LDS.
  // Instruction i of wave w (i < NA) fills tile rows 8 (NA w + i) .. +7 of a
  // stage; lane l lands at row 8 (NA w + i) + l/8, slot l%8, so it fetches the
  // K-chunk that the swizzle puts there, (l%8) ^ swz(row).  32-bit byte
  // offsets from the base (operands are < 4 GiB); rows of A past M re-read
  // row M-1 (never stored).
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p.A), 0, -1, 0x00020000);
  uint32_t a_src[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = 8 * (NA * wave + i) + (lane >> 3);
    int ga = m0 + row;
    ga = ga < M ? ga : M - 1;
    a_src[i] = (uint32_t)ga * (uint32_t)p.lda * 2u + (uint32_t)(((lane & 7) ^ swz(row)) << 4);
  }
  // quarter q (instructions AP q .. AP q + AP - 1) of A tile t into stage stg
  auto dma_a = [&](uint8_t* stg, int t, int q) {
    const int t_ = t < KT ? t : KT - 1;
    const uint32_t ko = (uint32_t)(kt0 + t_) * (BK * 2);
#pragma unroll
    for (int i = AP * q; i < AP * q + AP; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (lds_void_t*)(stg + 8 * (NA * wv + i) * ROW_BYTES), 16, a_src[i],
                                               ko, 0, 0);
  };

  // Residual epilogues of full tiles (RESID_SPLIT after the output
  // projection, RESID_PAIR after the down projection) with K tiles a multiple
  // of four: the ring loads of the last three K tiles, which would re-read the
  // last A tile, bring 64-row parts of the residual instead, one into each of
  // stages 0, 1, 2 (those of tiles KT - 4 .. KT - 2): rows 0..191 of R.  Wave w loads the 64
  // columns its own epilogue adds, into the 8 KiB of the stage its A loads
  // fill (rows of 128 bytes, the swizzle of A), so its epilogue reads them
  // after its own vmcnt wait, with no barrier.  Per quarter the same number of
  // loads as dma_a, so the ring's wait counts hold.
  constexpr bool kResLds = (EPI == EPI_RESID_SPLIT || EPI == EPI_RESID_PAIR) && BMT == 256 && !PART;
  const bool res_lds = kResLds && KT >= 4 && (KT & 3) == 0;
  // For the residual pair (R high, R2 low) the three parts are R rows 0..63,
  // R2 rows 0..63 and R rows 64..127.
  auto dma_r = [&](uint8_t* stg, int part, int q) {
    constexpr bool pair = EPI == EPI_RESID_PAIR;
    const void* base = pair && part == 1 ? p.R2 : p.R;
    const int r0 = pair ? (part == 2 ? 64 : 0) : 64 * part;
    const __amdgpu_buffer_rsrc_t rsr = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, -1, 0x00020000);
#pragma unroll
    for (int k = AP * q; k < AP * q + AP; ++k) {
      const int rs = 8 * k + (lane >> 3);                // row inside the 64-row part
      int row = m0 + r0 + rs;
      row = row < M ? row : M - 1;                       // rows past M are never stored
      const uint32_t col = (uint32_t)(n0 + 64 * wave + 8 * ((lane & 7) ^ swz(rs)));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsr, (lds_void_t*)(stg + wv * 8192 + k * 1024), 16,
                                               (uint32_t)row * (uint32_t)p.ldr * 2u + col * 2u, 0, 0, 0);
    }
  };

  // Fragment geometry: lane l holds row (l & 31) of a 32-row MFMA tile and
  // the 8 K values 16 s + 8 (l >> 5) .. +7 of K slice s.
  const int fr = lane & 31;
  const int fsw = swz(fr);
  const int fhalf = lane >> 5;
  const int a_row0 = fr * ROW_BYTES;

  // ---- B: straight into the operand registers -----------------------------
  // Column block j of the wave: lane l takes column wcol + 32 j + l%32.  In
  // the fragment-major weight, its operand of K slice s is the 16 bytes at
  // 16 l of the 1 KiB block (col / 32) * (K / 16) + s.
  const char* Bb = static_cast<const char*>(p.B);
  uint32_t b_off[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) b_off[j] = (uint32_t)((wcol >> 5) + j) * (uint32_t)(p.K >> 4) * 1024u + (uint32_t)lane * 16u;
  constexpr uint32_t B_TILE = 4096u;                // bytes of B per K tile and column block
  constexpr uint32_t B_SLICE = 1024u;

  f32x16_t acc[NI][2];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Software pipeline: tile t is multiplied out of LDS stage t%4 and B
  // register set t%2 while A tile t+3 streams into stage (t+3)%4 (the stage of
  // tile t-1) and B tile t+1 into the other register set.  The loop is
  // unrolled by four (stages) with a two-tile tail; K/64 is even for every
  // shape the bf16 path accepts.
  bf16x8_t bq0[2][4], bq1[2][4];
  bf16x8_t af[2][NI];

#define SEER_GLOAD_B(BQ, T, KS)                                                     \
  {                                                                                 \
    const int t_ = (T) < KT ? (T) : KT - 1;                                         \
    const char* bk_ = Bb + (size_t)(kt0 + t_) * B_TILE + (KS) * B_SLICE;            \
    _Pragma("unroll") for (int j = 0; j < 2; ++j)                                   \
      BQ[j][KS] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(bk_ + b_off[j])); \
  }
#define SEER_FLOAD(ST, KS, BUF)                                                     \
  {                                                                                 \
    const int chunk_ = ((2 * (KS) + fhalf) ^ fsw) << 4;                             \
    _Pragma("unroll") for (int i = 0; i < NI; ++i)                                  \
      af[BUF][i] = __builtin_bit_cast(bf16x8_t,                                     \
          *reinterpret_cast<const u32x4_t*>((ST) + a_row0 + i * 32 * ROW_BYTES + chunk_)); \
  }
  // One K tile of 4 slices x (NI x 2) MFMAs from stage SC.  Each slice is its
  // own scheduling region (sched_barrier fences) holding the fragment reads of
  // the next slice -- issued first, paired with the first MFMAs, so they have
  // the whole slice to land -- a quarter of A tile T+3 (into SF, the stage of
  // tile T-1, which every wave finished reading before the previous tile's
  // barrier) and slice s of B tile T+1.  After slice 2 one barrier publishes
  // A tile T+1 (stage SN) for slice 3's look-ahead read: before it, each wave
  // waits until its own loads of that tile (issued during tile T-2) have
  // landed -- at most the 7 slices of loads issued since may be in flight --
  // and until its LDS reads are done.  The barrier is bare (no fence): a
  // fence would also wait for the loads of tiles T+2 and T+3.
#define SEER_TILE_D(T, SC, SN, SF, BC, BNX, DMA)                                    \
  {                                                                                 \
    _Pragma("unroll") for (int ks = 0; ks < 4; ++ks) {                              \
      const int cur = ks & 1;                                                       \
      SEER_FLOAD(ks < 3 ? SC : SN, ks < 3 ? ks + 1 : 0, cur ^ 1);                   \
      DMA;                                                                          \
      SEER_GLOAD_B(BNX, (T) + 1, ks);                                               \
      _Pragma("unroll") for (int i = 0; i < NI; ++i)                                \
        _Pragma("unroll") for (int j = 0; j < 2; ++j)                               \
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(BC[j][ks], af[cur][i], acc[i][j], 0, 0, 0); \
      seer_slice_schedule<BMT>();                                                   \
      __builtin_amdgcn_sched_barrier(0);                                            \
      if (ks == 2) {                                                                \
        __builtin_amdgcn_s_waitcnt(waitcnt_imm(7 * (AP + 2), 0));                   \
        asm volatile("s_barrier" ::: "memory");                                     \
        __builtin_amdgcn_sched_barrier(0);                                          \
      }                                                                             \
    }                                                                               \
  }
#define SEER_TILE(T, SC, SN, SF, BC, BNX) SEER_TILE_D(T, SC, SN, SF, BC, BNX, dma_a(SF, (T) + 3, ks))

  // prologue: A tiles 0, 1, 2 into stages 0, 1, 2 and B tile 0 into set 0;
  // wait for all but tile 2 (its NA loads may stay in flight)
#pragma unroll
  for (int q = 0; q < 4; ++q) dma_a(st0, 0, q);
#pragma unroll
  for (int q = 0; q < 4; ++q) SEER_GLOAD_B(bq0, 0, q);
#pragma unroll
  for (int q = 0; q < 4; ++q) dma_a(st1, 1, q);
#pragma unroll
  for (int q = 0; q < 4; ++q) dma_a(st2, 2, q);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(NA, 15));
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  SEER_FLOAD(st0, 0, 0);
  int kt = 0;
  const int kt_ring = res_lds ? KT - 4 : KT;
  for (; kt + 4 <= kt_ring; kt += 4) {
    SEER_TILE(kt, st0, st1, st3, bq0, bq1);
    SEER_TILE(kt + 1, st1, st2, st0, bq1, bq0);
    SEER_TILE(kt + 2, st2, st3, st1, bq0, bq1);
    SEER_TILE(kt + 3, st3, st0, st2, bq1, bq0);
  }
  if constexpr (kResLds) {
    if (res_lds) {                                  // the last four K tiles
      SEER_TILE(kt, st0, st1, st3, bq0, bq1);
      SEER_TILE_D(kt + 1, st1, st2, st0, bq1, bq0, dma_r(st0, 0, ks));
      SEER_TILE_D(kt + 2, st2, st3, st1, bq0, bq1, dma_r(st1, 1, ks));
      SEER_TILE_D(kt + 3, st3, st0, st2, bq1, bq0, dma_r(st2, 2, ks));
      kt += 4;
    }
  }
  if (kt < KT) {                                   // K/64 = 2 mod 4
    SEER_TILE(kt, st0, st1, st3, bq0, bq1);
    SEER_TILE(kt + 1, st1, st2, st0, bq1, bq0);
  }
  // the loads past the last tile (clamped re-reads, or the residual parts)
  // land before the epilogue
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));
#undef SEER_GLOAD_B
#undef SEER_FLOAD
#undef SEER_TILE
#undef SEER_TILE_D

  // ---- K split: the fp32 sums of this split, row-major in the packed column
  // order of the weight (the finalize kernel applies the epilogue) ----------
  if constexpr (PART) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = m0 + i * 32 + fr;
      if (row < M) {
        float* prow = p.partial + ((size_t)split * (size_t)p.m_ub + (size_t)row) * (size_t)p.N + wcol + 4 * fhalf;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<f32x4_t*>(prow + 32 * j + 8 * q) =
                f32x4_t{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
      }
    }
    return;
  }

  // ---- epilogue -----------------------------------------------------------
  // The MFMAs take the B fragment as the matrix-core row operand, so tile
  // (i, j) accumulates the transposed 32x32 block: register r holds output
  // row m0 + 32 i + lane%32 and packed column wcol + 32 j + 8 (r/4) +
  // 4 (lane/32) + r%4.  Each lane owns one row and four consecutive columns
  // per register quad; lanes l and l+32 hold the two halves of each 8-column
  // group.  Stores and residual loads move 16 bytes (8 columns) per lane, and
  // one v_permlane32_swap per register pair deals them between the two
  // layouts.  For SWIGLU the gate/up tiles (j = 0, 1) sit in the same lane
  // and register; the near-zero count is a per-lane tally of its row, folded
  // over the lane pair.
  constexpr bool kGlu = (EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_COUNT);
  constexpr bool kRes = (EPI == EPI_RESID || EPI == EPI_RESID_SPLIT || EPI == EPI_RESID_PAIR);
  constexpr bool kPair = EPI == EPI_RESID_PAIR;
  constexpr bool kScale = EPI == EPI_SCALE || EPI == EPI_SCALE_ROPE;
  const int cq = 4 * fhalf;
  // Everything the epilogue reads besides the accumulators is requested ahead
  // of its use: the row scales of all 32-row blocks, and the residual columns
  // four blocks ahead.  Fetched block
  // by block between the stores, each block would wait out a full memory
  // latency behind the previous block's stores.  Residual word jt of a block
  // holds columns wcol + 16 jt + 8 (lane/32) .. +7 of the lane's row.
  constexpr int NRQ = (kPair ? 2 : 1) * 4;
  constexpr int RDEPTH = NI < 4 ? NI : 4;
  u32x4_t rq[RDEPTH][NRQ];
  const int colw = wcol + 8 * fhalf;
  auto fetch = [&](int i, u32x4_t* dst) {
    int row = m0 + i * 32 + fr;
    row = row < M ? row : M - 1;             // rows past M are never stored
    // row 32 (i % 2) + fr of a 64-row residual part in stage st; its swizzle
    // is that of fr
    auto lds_words = [&](const uint8_t* st, u32x4_t* w) {
      const uint8_t* sb = st + wv * 8192 + (32 * (i & 1) + fr) * ROW_BYTES;
#pragma unroll
      for (int jt = 0; jt < 4; ++jt) w[jt] = *reinterpret_cast<const u32x4_t*>(sb + (((fhalf + 2 * jt) ^ fsw) << 4));
    };
    if constexpr (kRes) {
      bool lds = false;
      if constexpr (kResLds) lds = res_lds && (kPair ? i < 4 : i < 6);
      if (lds) {
        lds_words(kPair ? (i < 2 ? st0 : st2) : (i < 2 ? st0 : i < 4 ? st1 : st2), dst);
      } else {
        const uint16_t* rb = R + (size_t)row * p.ldr + colw;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) dst[jt] = *reinterpret_cast<const u32x4_t*>(rb + 16 * jt);
      }
    }
    if constexpr (kPair) {
      bool lds = false;
      if constexpr (kResLds) lds = res_lds && i < 2;
      if (lds) {
        lds_words(st1, dst + 4);
      } else {
        const uint16_t* rb = static_cast<const uint16_t*>(p.R2) + (size_t)row * p.ldr + colw;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) dst[4 + jt] = *reinterpret_cast<const u32x4_t*>(rb + 16 * jt);
      }
    }
  };
  float rsv[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    int row = m0 + i * 32 + fr;
    row = row < M ? row : M - 1;
    rsv[i] = (kScale || EPI == EPI_ARGMAX || kGlu) ? p.rs[row] : 1.0f;
  }
  if constexpr (kRes) {
#pragma unroll
    for (int i = 0; i < RDEPTH; ++i) fetch(i, rq[i]);
  }
  // Output column of block j.  Below perm_col1 the packed weight holds each
  // 128-row head of q and k with its 32-row blocks in the order 0, 2, 1, 3, so
  // the wave's two blocks are features (32 h, 64 + 32 h) of one head, h = the
  // wave's 64-column half of the head: a rotary pair (c, c + 64) shares lane
  // and register.
  const bool perm = kScale && wcol < p.perm_col1;
  const int hsel = (wcol >> 6) & 1;
  int jcol[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) jcol[j] = perm ? (wcol & ~127) + 32 * (hsel + 2 * j) : wcol + 32 * j;
  constexpr bool kRope = EPI == EPI_SCALE_ROPE;
  const bool rope_on = kRope && wcol < p.rope_col1;
  int rpos[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) rpos[i] = 0;
  if (rope_on) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      int row = m0 + i * 32 + fr;
      row = row < M ? row : M - 1;
      rpos[i] = p.rope_pos[row];
    }
  }
  auto rope_block = [&](int i) {
    const double pos = (double)rpos[i];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        double rv = pos * p.rope_freq[32 * hsel + 8 * q + cq + e];
        rv -= floor(rv);
        const float t = (float)rv;            // revolutions in [0, 1)
        const float sn = __builtin_amdgcn_sinf(t), cs = __builtin_amdgcn_cosf(t);
        const float a = acc[i][0][4 * q + e], b = acc[i][1][4 * q + e];
        acc[i][0][4 * q + e] = a * cs - b * sn;
        acc[i][1][4 * q + e] = b * cs + a * sn;
      }
  };
  // V columns of the QKV projection are stored as fp16 (block-uniform)
  const bool to_f16 = kScale && p.f16_col0 > 0 && n0 >= p.f16_col0;

  // Stores: lanes l and l+32 hold the two 4-column halves of each 8-column
  // group of a row.  One v_permlane32_swap per packed register gives lane l
  // columns 8q..8q+7 and lane l+32 columns 8q+8..8q+15 of quads (q, q+1), so
  // every lane writes 16 contiguous bytes: half the store instructions of
  // 8-byte stores, which bound the epilogue.
  auto store_pair = [&](uint16_t* base, uint2 a, uint2 b) {
    const u32x2_t sx = __builtin_amdgcn_permlane32_swap(a.x, b.x, false, false);
    const u32x2_t sy = __builtin_amdgcn_permlane32_swap(a.y, b.y, false, false);
    *reinterpret_cast<u32x4_t*>(base) = u32x4_t{sx[0], sy[0], sx[1], sy[1]};
  };
  // the inverse: a 16-byte residual word back to the quads (q, q+1)
  auto split_pair = [&](u32x4_t w, uint2& a, uint2& b) {
    const u32x2_t sx = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
    const u32x2_t sy = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
    a.x = sx[0]; a.y = sy[0];
    b.x = sx[1]; b.y = sy[1];
  };
  auto add_bf4 = [](float* v, uint2 r) {
    v[0] += __uint_as_float(r.x << 16);
    v[1] += __uint_as_float(r.x & 0xffff0000u);
    v[2] += __uint_as_float(r.y << 16);
    v[3] += __uint_as_float(r.y & 0xffff0000u);
  };

  // largest magnitude this lane stored as fp16 (the range check of V)
  float f16_max = 0.0f;
  // One 32-row block of the non-GLU epilogues, straight-line for one output
  // type (F16 is the type of the whole block).
  auto store_block = [&](auto f16_tag, int i, const u32x4_t* rr) {
    constexpr bool F16 = decltype(f16_tag)::value;
    const int row = m0 + i * 32 + fr;
    if (row >= M) return;
    const float sc = rsv[i];
    uint16_t* crow = C + (size_t)row * p.ldc + 8 * fhalf;
    uint16_t* cw2 = EPI == EPI_RESID_SPLIT ? static_cast<uint16_t*>(p.C2) + (size_t)row * p.ldc + colw : nullptr;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      uint2 rv[4], rv2[4];
      if constexpr (kRes) {
        split_pair(rr[2 * j], rv[0], rv[1]);
        split_pair(rr[2 * j + 1], rv[2], rv[3]);
      }
      if constexpr (kPair) {
        split_pair(rr[4 + 2 * j], rv2[0], rv2[1]);
        split_pair(rr[4 + 2 * j + 1], rv2[2], rv2[3]);
      }
      uint2 pk[4], lo[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];
        if constexpr (kScale) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] *= sc;
        }
        if constexpr (kRes) add_bf4(v, rv[q]);
        if constexpr (kPair) add_bf4(v, rv2[q]);
        if constexpr (F16) {
#pragma unroll
          for (int e = 0; e < 4; ++e) f16_max = fmaxf(f16_max, fabsf(v[e]));
        }
        pk[q].x = F16 ? pack_h2(v[0], v[1]) : pack_bf2(v[0], v[1]);
        pk[q].y = F16 ? pack_h2(v[2], v[3]) : pack_bf2(v[2], v[3]);
        if constexpr (EPI == EPI_RESID_SPLIT) {
          // v - bf16(v) is exact in fp32; its bf16 rounding leaves ~2^-17 of v
          lo[q].x = pack_bf2(v[0] - __uint_as_float(pk[q].x << 16), v[1] - __uint_as_float(pk[q].x & 0xffff0000u));
          lo[q].y = pack_bf2(v[2] - __uint_as_float(pk[q].y << 16), v[3] - __uint_as_float(pk[q].y & 0xffff0000u));
        }
      }
      store_pair(crow + jcol[j], pk[0], pk[1]);
      store_pair(crow + jcol[j] + 16, pk[2], pk[3]);
      if constexpr (EPI == EPI_RESID_SPLIT) {
        store_pair(cw2 + 32 * j, lo[0], lo[1]);
        store_pair(cw2 + 32 * j + 16, lo[2], lo[3]);
      }
    }
  };

  // Rotated q/k waves take their own straight-line path (bf16 stores), so
  // that no accumulator values from rotated and unrotated paths meet.
  if constexpr (kRope) {
    if (rope_on) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        rope_block(i);
        store_block(std::false_type{}, i, rq[0]);
      }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int row = m0 + i * 32 + fr;
    const bool ok = row < M;
    if constexpr (kGlu) {
      const float sc = rsv[i];
      int nz = 0;
      uint2 pk[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float a[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          a[e] = silu(acc[i][0][4 * q + e] * sc) * (acc[i][1][4 * q + e] * sc);
          // |a| < eps as the sign bit of |a| - eps: rounding keeps the sign of a
          // difference and equality gives +0 (no compare, no SGPR hazard)
          if constexpr (EPI == EPI_SWIGLU_COUNT) nz += __float_as_uint(fabsf(a[e]) - p.eps) >> 31;
        }
        pk[q].x = pack_bf2(a[0], a[1]);
        pk[q].y = pack_bf2(a[2], a[3]);
      }
      // the swaps are wave-wide: every lane takes part, rows past M store nothing
      uint16_t* cw = C + (size_t)row * p.ldc + (wcol >> 1) + 8 * fhalf;
      const u32x2_t s0x = __builtin_amdgcn_permlane32_swap(pk[0].x, pk[1].x, false, false);
      const u32x2_t s0y = __builtin_amdgcn_permlane32_swap(pk[0].y, pk[1].y, false, false);
      const u32x2_t s1x = __builtin_amdgcn_permlane32_swap(pk[2].x, pk[3].x, false, false);
      const u32x2_t s1y = __builtin_amdgcn_permlane32_swap(pk[2].y, pk[3].y, false, false);
      if (ok) {
        *reinterpret_cast<u32x4_t*>(cw) = u32x4_t{s0x[0], s0y[0], s0x[1], s0y[1]};
        *reinterpret_cast<u32x4_t*>(cw + 16) = u32x4_t{s1x[0], s1y[0], s1x[1], s1y[1]};
      }
      if constexpr (EPI == EPI_SWIGLU_COUNT) {
        nz += __shfl_xor(nz, 32, kWave);
        if (ok && fhalf == 0) atomicAdd(p.cnt + row, nz);
      }
    } else if constexpr (EPI == EPI_ARGMAX) {
      // the lane's 32 columns of its row in increasing order, so a strict >
      // keeps the smallest column among equal maxima; then the lane pair
      const float sc = rsv[i];
      const int cb = wcol + cq;
      float m = -INFINITY;
      int a = cb;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float v = acc[i][j][4 * q + e] * sc;
            if (v > m) { m = v; a = cb + 32 * j + 8 * q + e; }
          }
      float sum = 0.0f;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += __expf(acc[i][j][r] * sc - m);
      const float m2 = __shfl_xor(m, 32, kWave);
      const float s2 = __shfl_xor(sum, 32, kWave);
      const int a2 = __shfl_xor(a, 32, kWave);
      const float mm = fmaxf(m, m2);
      const float st = sum * __expf(m - mm) + s2 * __expf(m2 - mm);
      const int at = (m2 > m || (m2 == m && a2 < a)) ? a2 : a;
      if (ok && fhalf == 0) {
        ArgmaxPartial* dst = static_cast<ArgmaxPartial*>(p.C) + (size_t)row * p.ldc + (wcol >> 6);
        *reinterpret_cast<u32x4_t*>(dst) = u32x4_t{__float_as_uint(mm), __float_as_uint(st), (uint32_t)at, 0u};
      }
    } else {
      const u32x4_t* rr = rq[i % RDEPTH];
      if (kScale && to_f16)
        store_block(std::true_type{}, i, rr);
      else
        store_block(std::false_type{}, i, rr);
      // the block RDEPTH ahead goes into the buffer just used
      if constexpr (kRes) {
        if (i + RDEPTH < NI) fetch(i + RDEPTH, rq[i % RDEPTH]);
      }
    }
  }
  // V beyond fp16's finite range was stored rounded (+-65504 or +-inf): report
  // it (rare; one atomic per offending lane)
  if constexpr (kScale) {
    if (to_f16 && p.status && f16_max > 65504.0f) atomicOr(p.status, SEER_STATUS_V_RANGE);
  }
}

// Units of work: the 256x256 tiles, except that when the tiles leave a last
// round of r < n_units/2 tiles on the n_units workgroups that run at once,
// each of those r tiles becomes two 128x256 halves (disjoint outputs, no
// reduction), so the last round keeps twice as many CUs busy; a last tile
// row of at most 128 rows is computed as half tiles only.  Tile geometry
// follows the real row count read on the device (or the row-tile list of
// p.mtiles); surplus blocks of the upper-bound grid, and halves that start
// past the last row, exit at once.
template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmParams p) {
  // the four stages of the A ring, each its own array: the compiler then
  // orders fragment reads of one stage only after the loads into that stage
  __shared__ __attribute__((aligned(1024))) uint8_t st0[256 * ROW_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[256 * ROW_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t st2[256 * ROW_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t st3[256 * ROW_BYTES];
  const int M = rows_from(p.m_ptr, p.m_ub);
  const int tiles_m = p.mtiles ? p.mtiles[0] : (M + 255) / 256;
  const int tiles_n = p.N / 256;
  // A last tile row that holds at most 128 rows runs as single half tiles
  // (their second halves would hold no row); the full tiles are those of the
  // other rows.
  const bool half_last = !p.mtiles && tiles_m > 0 && M - 256 * (tiles_m - 1) <= 128;
  const int tiles_mf = tiles_m - (half_last ? 1 : 0);
  const int nfull = tiles_mf * tiles_n;
  const int nlast = half_last ? tiles_n : 0;
  int full = nfull;
  if (p.n_units > 0) {
    const int rem = nfull % p.n_units;
    if (2 * rem + nlast <= p.n_units) full = nfull - rem;
  }
  const int nsplit = 2 * (nfull - full);           // halves of the tiles past `full`
  const int u = blockIdx.x;
  const int KT = p.K / BK;
  int tm, tn;
  if (u >= full + nsplit + nlast) return;
  if (u < full) {
    raster(xcd_remap(u, full), tiles_mf, tiles_n, tm, tn);
    if (p.mtiles) tm = p.mtiles[1 + tm];
    gemm_tile<EPI, 256>(p, st0, st1, st2, st3, M, tm * 256, tn * 256, 0, KT);
  } else {
    const int v = u - full;
    int m0;
    if (v < nsplit) {
      raster(full + (v >> 1), tiles_mf, tiles_n, tm, tn);
      if (p.mtiles) tm = p.mtiles[1 + tm];
      m0 = tm * 256 + (v & 1) * 128;
    } else {
      tn = v - nsplit;
      m0 = (tiles_m - 1) * 256;
    }
    if (m0 >= M) return;
    gemm_tile<EPI, 128>(p, st0, st1, st2, st3, M, m0, tn * 256, 0, KT);
  }
}

// K-split launches (a kernel of its own, so that the register allocation of
// the main kernel does not change): unit u computes split u % S of tile u / S
// over K tiles [s KT/S, (s+1) KT/S) and stores its fp32 sums; the host chose S
// so that KT/S is even and the units fit one round.
template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_split_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t st0[256 * ROW_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[256 * ROW_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t st2[256 * ROW_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t st3[256 * ROW_BYTES];
  const int M = rows_from(p.m_ptr, p.m_ub);
  const int tiles_m = p.mtiles ? p.mtiles[0] : (M + 255) / 256;
  const int tiles_n = p.N / 256;
  const int S = p.k_splits;
  const int u = blockIdx.x;
  if (u >= tiles_m * tiles_n * S) return;
  const int tile = u / S, sp = u - tile * S;
  const int kts = p.K / BK / S;
  int tm, tn;
  raster(tile, tiles_m, tiles_n, tm, tn);
  if (p.mtiles) tm = p.mtiles[1 + tm];
  gemm_tile<EPI, 256, true>(p, st0, st1, st2, st3, M, tm * 256, tn * 256, sp * kts, kts, sp);
}

// The epilogue of a K-split launch: for row r < M and 8 consecutive output
// columns per thread, the splits' fp32 sums are added in split order (the
// result does not depend on timing) and the launch's epilogue is applied to
// them exactly as the GEMM applies it to its accumulators.  Partial column
// order is the packed weight's: SWIGLU takes gate and up from packed columns
// 64 k + e and 64 k + 32 + e for output column 32 k + e; SCALE's head-permuted
// q/k columns go back to head order.  With a row-tile list, thread rows run
// over the listed tiles only.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_finalize_kernel(GemmParams p) {
  constexpr bool kGlu = EPI == EPI_SWIGLU;
  const int M = rows_from(p.m_ptr, p.m_ub);
  const int groups = kGlu ? p.N / 16 : p.N / 8;          // 8-column output groups per row
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const int vrow = (int)(idx / groups);
  const int g = (int)(idx - (long long)vrow * groups);
  int row = vrow;
  if (p.mtiles) {
    if ((vrow >> 8) >= p.mtiles[0]) return;
    row = p.mtiles[1 + (vrow >> 8)] * 256 + (vrow & 255);
  }
  if (row >= M) return;
  const int S = p.k_splits;
  auto sum8 = [&](int col, float* v) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = 0.0f;
    for (int sp = 0; sp < S; ++sp) {
      const float* src = p.partial + ((size_t)sp * (size_t)p.m_ub + (size_t)row) * (size_t)p.N + col;
      const f32x4_t a = *reinterpret_cast<const f32x4_t*>(src);
      const f32x4_t b = *reinterpret_cast<const f32x4_t*>(src + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] += a[e];
        v[4 + e] += b[e];
      }
    }
  };
  auto pack8_bf = [](const float* v) {
    return u32x4_t{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7])};
  };
  auto add8_bf = [](float* v, u32x4_t r) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] += __uint_as_float(r[e] << 16);
      v[2 * e + 1] += __uint_as_float(r[e] & 0xffff0000u);
    }
  };
  float v[8];
  if constexpr (kGlu) {
    const int oc = 8 * g, kb = oc >> 5, e0 = oc & 31;
    float u[8];
    sum8(64 * kb + e0, v);
    sum8(64 * kb + 32 + e0, u);
    const float sc = p.rs[row];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = silu(v[e] * sc) * (u[e] * sc);
    *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.C) + (size_t)row * p.ldc + oc) = pack8_bf(v);
  } else {
    const int pc = 8 * g;
    sum8(pc, v);
    if constexpr (EPI == EPI_SCALE) {
      int oc = pc;
      if (pc < p.perm_col1) {
        const int hsel = (pc >> 6) & 1, j = (pc >> 5) & 1;
        oc = (pc & ~127) + 32 * (hsel + 2 * j) + (pc & 31);
      }
      const float sc = p.rs[row];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] *= sc;
      uint16_t* dst = static_cast<uint16_t*>(p.C) + (size_t)row * p.ldc + oc;
      if (p.f16_col0 > 0 && oc >= p.f16_col0) {
        float mx = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, fabsf(v[e]));
        *reinterpret_cast<u32x4_t*>(dst) =
            u32x4_t{pack_h2(v[0], v[1]), pack_h2(v[2], v[3]), pack_h2(v[4], v[5]), pack_h2(v[6], v[7])};
        if (p.status && mx > 65504.0f) atomicOr(p.status, SEER_STATUS_V_RANGE);
      } else {
        *reinterpret_cast<u32x4_t*>(dst) = pack8_bf(v);
      }
    } else {
      // residual adds: v + R (RESID_SPLIT: stored as the bf16 pair hi, lo) or
      // v + R + R2 (RESID_PAIR)
      add8_bf(v, *reinterpret_cast<const u32x4_t*>(static_cast<const uint16_t*>(p.R) + (size_t)row * p.ldr + pc));
      if constexpr (EPI == EPI_RESID_PAIR)
        add8_bf(v, *reinterpret_cast<const u32x4_t*>(static_cast<const uint16_t*>(p.R2) + (size_t)row * p.ldr + pc));
      const u32x4_t hi = pack8_bf(v);
      *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.C) + (size_t)row * p.ldc + pc) = hi;
      if constexpr (EPI == EPI_RESID_SPLIT) {
        float lo[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          lo[2 * e] = v[2 * e] - __uint_as_float(hi[e] << 16);
          lo[2 * e + 1] = v[2 * e + 1] - __uint_as_float(hi[e] & 0xffff0000u);
        }
        *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.C2) + (size_t)row * p.ldc + pc) = pack8_bf(lo);
      }
    }
  }
}

// K splits for a launch of `tiles` 256x256 tiles: the most splits (<= 16)
// whose units fit one round on the n_units workgroups that run at once, with
// an even number of 64-wide K tiles per split (the main loop's unroll) and
// partials that fit the scratch -- used only when that is at least 3 and the
// epilogue can be split.  Two splits gain nothing over the half-height tiles
// of the unsplit launch and cost the finalize pass (measured: the prefix-
// cached B=16 step 0.745 -> 0.763 ms); at 3 and more the launch takes a
// fraction of one tile's time (the B=1 cached step 0.359 -> 0.198 ms).
static int k_splits_for(int epi, const GemmParams& p, int tiles, int tiles_m) {
  const bool splittable = epi == EPI_SCALE || epi == EPI_RESID_SPLIT || epi == EPI_RESID_PAIR || epi == EPI_SWIGLU;
  if (!splittable || !p.partial || p.n_units <= 0 || tiles < 1) return 1;
  const int KT = p.K / BK;
  int S = p.n_units / tiles;
  S = S < 16 ? S : 16;
  while (S > 1 && (KT % (2 * S) != 0 || (size_t)S * (size_t)tiles_m * 256u * (size_t)p.N * 4u > p.partial_bytes)) --S;
  return S >= 3 ? S : 1;
}

int launch_gemm_bf16(int epi, const GemmParams& p_in, hipStream_t s) {
  GemmParams p = p_in;
  // the head permutation and the rotary pairs work on whole 128-wide heads of
  // the SCALE epilogues, and rotation needs the permuted layout
  const bool scale = epi == EPI_SCALE || epi == EPI_SCALE_ROPE;
  if (p.perm_col1 && (!scale || p.perm_col1 % 128 != 0)) return -1;
  if ((epi == EPI_SCALE_ROPE) != (p.rope_pos != nullptr)) return -1;
  if (p.rope_pos && (!p.rope_freq || p.rope_col1 % 128 != 0 || p.rope_col1 > p.perm_col1)) return -1;
  const int tiles_m = (p.m_ub + 255) / 256;
  const int tiles_n = p.N / 256;
  p.k_splits = k_splits_for(epi, p, tiles_m * tiles_n, tiles_m);
  // the split last round adds at most n_units / 2 units; a K split has
  // k_splits units per tile
  dim3 grid(p.k_splits > 1 ? tiles_m * tiles_n * p.k_splits : tiles_m * tiles_n + (p.n_units > 0 ? p.n_units / 2 : 0)),
      block(NT);
  if (p.k_splits > 1) {
    switch (epi) {
      case EPI_SCALE: hipLaunchKernelGGL(gemm_bf16_split_kernel<EPI_SCALE>, grid, block, 0, s, p); break;
      case EPI_RESID_SPLIT: hipLaunchKernelGGL(gemm_bf16_split_kernel<EPI_RESID_SPLIT>, grid, block, 0, s, p); break;
      case EPI_RESID_PAIR: hipLaunchKernelGGL(gemm_bf16_split_kernel<EPI_RESID_PAIR>, grid, block, 0, s, p); break;
      case EPI_SWIGLU: hipLaunchKernelGGL(gemm_bf16_split_kernel<EPI_SWIGLU>, grid, block, 0, s, p); break;
      default: return -1;
    }
  } else switch (epi) {
    case EPI_SCALE: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SCALE>, grid, block, 0, s, p); break;
    case EPI_SCALE_ROPE: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SCALE_ROPE>, grid, block, 0, s, p); break;
    case EPI_SWIGLU: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU>, grid, block, 0, s, p); break;
    case EPI_SWIGLU_COUNT:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU_COUNT>, grid, block, 0, s, p); break;
    case EPI_RESID_SPLIT:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID_SPLIT>, grid, block, 0, s, p); break;
    case EPI_RESID_PAIR:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID_PAIR>, grid, block, 0, s, p); break;
    case EPI_ARGMAX: hipLaunchKernelGGL(gemm_bf16_kernel<EPI_ARGMAX>, grid, block, 0, s, p); break;
    default: return -1;
  }
  if (p.k_splits > 1) {
    const long long groups = (long long)p.m_ub * (epi == EPI_SWIGLU ? p.N / 16 : p.N / 8);
    dim3 fgrid((unsigned)((groups + 255) / 256)), fblock(256);
    switch (epi) {
      case EPI_SCALE: hipLaunchKernelGGL(gemm_finalize_kernel<EPI_SCALE>, fgrid, fblock, 0, s, p); break;
      case EPI_RESID_SPLIT: hipLaunchKernelGGL(gemm_finalize_kernel<EPI_RESID_SPLIT>, fgrid, fblock, 0, s, p); break;
      case EPI_RESID_PAIR: hipLaunchKernelGGL(gemm_finalize_kernel<EPI_RESID_PAIR>, fgrid, fblock, 0, s, p); break;
      case EPI_SWIGLU: hipLaunchKernelGGL(gemm_finalize_kernel<EPI_SWIGLU>, fgrid, fblock, 0, s, p); break;
      default: return -1;
    }
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace seer
