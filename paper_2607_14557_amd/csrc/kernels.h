// Internal launchers of the Seer layer library (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "seer.h"

namespace seer {

// SCALE: C = acc * rs[r]; SCALE_ROPE: SCALE with the rotary embedding of the
// columns < rope_col1 (bf16 only); RESID: C = R + acc; SWIGLU(_COUNT): gate/up pairs;
// RESID_SPLIT: v = R + acc, C = bf16(v), C2 = bf16(v - C) (bf16 only);
// RESID_PAIR: C = bf16(R + R2 + acc) (bf16 only);
// ARGMAX: no output matrix; per row and 64-column block of l = acc * rs[r],
// the partial {max, sum exp(l - max), argmax column} (bf16 only, see
// ArgmaxPartial).
enum Epilogue {
  EPI_SCALE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_SWIGLU_COUNT = 3,
  EPI_RESID_SPLIT = 4, EPI_RESID_PAIR = 5, EPI_ARGMAX = 6, EPI_SCALE_ROPE = 7
};

// One row's partial over 64 columns (EPI_ARGMAX): C is ArgmaxPartial[M][N/64].
struct ArgmaxPartial {
  float max;
  float sum;     // sum of exp(l - max) over the block
  int arg;       // smallest column reaching max
  int pad;
};

// C[M,N] = A[M,K] * B[N,K]^T with a fused epilogue.  M is read on the device
// from m_ptr (clamped to m_ub, the bound the grid is sized from).
struct GemmParams {
  const void* A;
  const void* B;
  void* C;
  const void* R;      // residual rows (RESID*), same element type as C
  void* C2;           // low part of the output, same layout as C (RESID_SPLIT)
  const void* R2;     // low part of the residual, same layout as R (RESID_PAIR)
  const float* rs;    // per-row scale (SCALE, SWIGLU*)
  int* cnt;           // per-row near-zero count (SWIGLU_COUNT)
  float eps;
  const int* m_ptr;
  int m_ub;
  int N;
  int K;
  int lda, ldb, ldc, ldr;
  // fp32 SwiGLU only: the up-projection weight as a second [N, K] operand
  const void* B2;
  // bf16 SCALE only: output columns >= f16_col0 are stored as fp16 (the V
  // third of the QKV projection); 0 means none
  int f16_col0;
  // bf16 only: workgroups that run at once (one per CU).  When the 256x256
  // tiles leave a last round of r <= n_units / 2 tiles, those r tiles run as
  // 2 r halves of 128x256 (split along rows).  0 disables the split.
  int n_units;
  // bf16 SCALE_ROPE only (and required there): rotary embedding of output
  // columns < rope_col1 (whole 128-wide heads): row r's pair (c, c + 64) of
  // each head is rotated by 2 pi * frac(rope_pos[r] * rope_freq[c % 64])
  const int* rope_pos;
  const double* rope_freq;
  int rope_col1;
  // bf16 SCALE(_ROPE) only: output columns < perm_col1 (whole 128-wide heads) come
  // from weight rows packed in head-block order 0, 2, 1, 3 (qk_packed_row)
  // and are stored back in head order; 0 means none.  rope_col1 <= perm_col1.
  int perm_col1;
  // bf16 SCALE(_ROPE) only, optional: status word that receives
  // SEER_STATUS_V_RANGE (atomic OR) when a column stored as fp16 had a
  // magnitude above fp16's largest finite value
  int* status;
  // bf16 SCALE, RESID_SPLIT, RESID_PAIR and SWIGLU, optional: scratch for
  // fp32 partial tiles (partial_bytes bytes).  A launch whose 256x256 tiles
  // fill at most a third of the n_units workgroups that run at once splits K
  // over k_splits units per tile: each stores its fp32 partial sums, and a
  // second kernel adds the splits in order and applies the epilogue.  The
  // launcher sets k_splits; callers leave it 0.
  float* partial;
  size_t partial_bytes;
  int k_splits;
  // bf16, optional: the 256-row tiles to compute.  mtiles[0] = their number,
  // mtiles[1 ..] = their indices t (rows 256 t .. 256 t + 255) in increasing
  // order, written on the device (launch_kept_tiles); the launch covers them
  // as if they were consecutive and leaves the other rows of C untouched.
  // Null: every row.
  const int* mtiles;
};

// Weight layout of the bf16 GEMM's B operand ("fragment-major"): element
// (n, k) of a [N, K] matrix (N % 32 == 0, K % 16 == 0) sits at this index, so
// the 32x32x16 MFMA operand of 32 columns and one 16-wide K slice is one
// 1 KiB block holding lane l's 8 values (column n % 32 = l % 32, k % 16 in
// 8 (l / 32) .. +7) at 16 l bytes.
__host__ __device__ inline size_t frag_b_index(size_t n, size_t k, size_t K) {
  return ((n / 32) * (K / 16) + k / 16) * 512 + (((k % 16) / 8) * 32 + n % 32) * 8 + k % 8;
}

// Packed q/k row r (r < 2 d) holds weight row qk_packed_row(r): within each
// 128-row head the 32-row blocks are in the order 0, 2, 1, 3 (an involution),
// so one wave's 64 output columns hold the rotary pairs (c, c + 64) of a head.
__host__ __device__ inline size_t qk_packed_row(size_t r) {
  const size_t b = (r >> 5) & 3;
  const size_t nb = b == 1 ? 2 : (b == 2 ? 1 : b);
  return (r & ~(size_t)127) + nb * 32 + (r & 31);
}

// bf16 operands; requires N % 256 == 0, K % 128 == 0, 16-byte aligned rows.
// B is fragment-major (frag_b_index); ldb is unused.
// For SWIGLU*, N is the packed 2*I and C has I columns.
int launch_gemm_bf16(int epi, const GemmParams& p, hipStream_t s);

// fp32 operands, any N and K.  For SWIGLU*, B = Wg, B2 = Wu, both [N=I, K].
int launch_gemm_f32(int epi, const GemmParams& p, hipStream_t s);

// Row positions and rotary frequencies for the rotary embedding of q and k:
// pos[r] = r - cu[b] + (cu_kv ? cu_kv[b+1] - cu_kv[b] : 0) for the sequence b
// holding row r < M, and freq[j] = theta^(-2 j / head_dim) / (2 pi) (in
// revolutions per position) for j < head_dim / 2.
struct RopeArgs {
  const int* cu;
  int B;
  const int* cu_kv;
  int* pos;
  double* freq;
  float theta;
  int head_dim;
};

// inv_rms[r] = 1 / sqrt(mean_j x[r,j]^2 + eps) for r < M; with rope, also
// the rotary positions and frequencies above.
int launch_rms_inv(bool bf16, const void* x, int ld, int d, const int* m_ptr, int m_ub,
                   float eps, float* out, hipStream_t s, const RopeArgs* rope = nullptr);

// fp32: rotate the q and k columns of qkv ([M, 3d]) in place with the
// positions and frequencies written by launch_rms_inv.
int launch_rope_f32(float* qkv, int d, int n_heads, int head_dim, const int* m_ptr, int m_ub,
                    const int* pos, const double* freq, hipStream_t s);

struct AttnParams {
  const void* qkv;       // [T, 3d]: q | k | v, head h at columns h*dh of each
  void* out;             // [T, d]
  const int* cu;         // [B+1]
  const int* used;       // [B] or null
  int B;
  int d;
  int n_heads;
  int head_dim;
  int rows_ub;           // bound on cu[B] (sizes the grid)
  float scale;           // 1/sqrt(head_dim)
  // optional cached prefix keys/values: sequence b's queries also attend to
  // cache rows [cu_kv[b], cu_kv[b+1]) of kv ([rows, 2d]: K | V, the element
  // types of the K and V thirds of qkv), ahead of its own keys; null: none
  const void* kv;
  const int* cu_kv;
};

int launch_attn_bf16(const AttnParams& p, hipStream_t s);
int launch_attn_f32(const AttnParams& p, hipStream_t s);

// Zero an int32 array of n entries.
int launch_zero_i32(int* p, int n, hipStream_t s);

struct DetectParams {
  const int* cnt;
  const int* cu;
  const int* win_off;
  const int* win_len;
  int B;
  int d_ff;
  int tau_num, tau_den, gamma_num, gamma_den, lookahead;
  int* boundary;
  int* keep_len;
};
int launch_detect(const DetectParams& p, hipStream_t s);

// The 256-row tiles of a packed batch that hold rows the compaction keeps:
// row r of sequence b is kept when r - cu[b] < win_off[b] + keep_len[b]
// (keep_len clamped to [0, win_len[b]], the sum to the sequence's length).
// map[0] = the number of such tiles t < ceil(min(cu[B], rows_ub) / 256),
// map[1 ..] = the tiles in increasing order (the mtiles of GemmParams); map
// holds 1 + ceil(rows_ub / 256) entries.  One workgroup.
struct KeptTilesParams {
  const int* cu;
  const int* win_off;
  const int* win_len;
  const int* keep_len;
  int B;
  int rows_ub;
  int* map;
};
int launch_kept_tiles(const KeptTilesParams& p, hipStream_t s);

constexpr int kRepackMaxBatch = 1024;
constexpr int kRepackMaxBuffers = 4;

struct RepackParams {
  const uint8_t* src[kRepackMaxBuffers];
  uint8_t* dst[kRepackMaxBuffers];
  int n_buffers;
  const int* cu_src;
  const int* win_off;
  const int* win_len;
  const int* keep_len;
  int B;
  int policy;
  int tau_num, tau_den;
  int granule;
  int row_bytes;
  int dst_capacity_rows;
  int* cu_dst;
  int* seqused;
  int* route;
  int* ctrl_dev;    // seer_route_ctrl as int[16]
  int* ctrl_host;
  bool window_only; // copy only the kept window rows (no prefix rows)
};
int launch_repack(const RepackParams& p, hipStream_t s);

// K | V columns of the prefix rows of each sequence, from the qkv rows of a
// layer call (row stride 3 d elements) into a cache ([rows, 2 d]).
struct KvExportParams {
  const uint8_t* qkv;
  const int* cu;        // [B+1] rows of the layer call
  const int* cu_kv;     // [B+1] cache rows; sequence b's prefix has cu_kv[b+1] - cu_kv[b] rows
  uint8_t* dst;
  int B;
  int d;
  int es;               // bytes per element
  int rows_ub;          // rows of the qkv region
};
int launch_kv_export(const KvExportParams& p, int kv_rows_ub, hipStream_t s);

// Per row r < M (M from m_ptr): merge the n_part ArgmaxPartial entries into
// the prediction (smallest column among equal maxima) and its softmax
// probability 1 / sum_p sum_p exp(max_p - max).
int launch_argmax_reduce(const void* partials, int n_part, const int* m_ptr, int m_ub, int* pred, float* conf,
                         hipStream_t s);

// Remasking step (two launches: the decision, one workgroup per sequence,
// then the rows) over rows [cu[b], cu[b+1]) of sequence b, the first used[b]
// real: commit the ceil(n / steps_left) most confident masked
// positions (tokens == -1), ties to the smaller position, then write the next
// input rows: emb[token] if committed, x0 row if masked, zero past used.
struct RemaskParams {
  const int* cu;
  const int* used;
  int B;
  int max_used;          // bound on used[b] (clamps it)
  int steps_left;
  const int* pred;
  const float* conf;
  int* tokens;
  const uint16_t* x0;    // [rows, d] bf16
  const uint16_t* emb;   // [vocab, d] bf16
  int vocab;
  uint16_t* x_next;      // [rows, d] bf16
  int d;
};
int launch_remask(const RemaskParams& p, hipStream_t s);

struct PrepackParams {
  const void* wq; const void* wk; const void* wv; const void* wo;
  const void* wg; const void* wu; const void* wd;
  const float* g1; const float* g2;
  void* dst;
  int d, d_ff;
  bool bf16;
};
// Offsets (in elements) of the packed blocks.
struct PackedLayout {
  size_t qkv, o, gu, dn, total_bytes;
};
PackedLayout packed_layout(int d, int d_ff, bool bf16);
int launch_prepack(const PrepackParams& p, hipStream_t s);

// Copy a row-major bf16 matrix src [N, K] (N % 32 == 0, K % 16 == 0) to dst
// in the fragment-major order of frag_b_index.
int launch_pack_frag(const void* src, int N, int K, void* dst, hipStream_t s);

}  // namespace seer
